// Integer code intervals of the estimate (the coding of Alg. 1, line 9).
// For logits z[256] of a window: m = max z, d_s = (m - z_s) log2(e) in float32
// (two correctly rounded operations, no contraction), u_s = trunc(256 d_s +
// 1/2) capped at 32*256 - 1, w_s = T[u_s mod 256] >> (u_s div 256) with
// T[j] = round(2^31 2^(-j/256)), and freq_s = 1 + 65280 w_s div sum w.  Past
// d_s the arithmetic is exact, so the encoder's and the decoder's launches
// (and any implementation of these steps) give the same frequencies.
#include <cmath>

#include "codec.h"

namespace {
struct QuantTab {
  uint32_t t[256];
};

// one wave per window, lane l holds bytes 4l .. 4l+3
__global__ __launch_bounds__(256) void k_quantize(const float* __restrict__ z, int64_t n, uint16_t* __restrict__ freq,
                                                  QuantTab tab) {
  const int lane = threadIdx.x & 63;
  const int64_t w = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (w >= n) return;  // whole waves
  const float4 v = *reinterpret_cast<const float4*>(z + w * 256 + 4 * lane);
  float m = fmaxf(fmaxf(v.x, v.y), fmaxf(v.z, v.w));
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) m = fmaxf(m, __shfl_xor(m, o));
  const float zz[4] = {v.x, v.y, v.z, v.w};
  uint32_t wt[4];
  uint64_t S = 0;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const float d = __fmul_rn(__fsub_rn(m, zz[r]), 1.4426950408889634f);
    int u = QMAX;
    if (d < 32.0f) u = min((int)__fadd_rn(__fmul_rn(d, 256.0f), 0.5f), QMAX);
    wt[r] = tab.t[u & 255] >> (u >> 8);
    S += wt[r];
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) S += (uint64_t)__shfl_xor((long long)S, o);
  uint16_t f[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) f[r] = (uint16_t)(1 + ((uint64_t)wt[r] * QSPREAD) / S);
  *reinterpret_cast<uint2*>(freq + w * 256 + 4 * lane) =
      make_uint2((uint32_t)f[0] | ((uint32_t)f[1] << 16), (uint32_t)f[2] | ((uint32_t)f[3] << 16));
}
// column col of n rows of stride bytes from n contiguous bytes
__global__ __launch_bounds__(256) void k_put_column(const uint8_t* __restrict__ src, int64_t n,
                                                    uint8_t* __restrict__ dst, int64_t stride, int64_t col) {
  const int64_t b = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (b < n) dst[b * stride + col] = src[b];
}
}  // namespace

void launch_put_column(const uint8_t* src, int64_t n, uint8_t* dst, int64_t stride, int64_t col, hipStream_t s) {
  if (n <= 0) return;
  hipLaunchKernelGGL(k_put_column, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, src, n, dst, stride, col);
}

const uint32_t* quant_table() {
  static const QuantTab tab = [] {
    QuantTab t;
    // 2^(-j/256) in extended precision, rounded to the nearest integer at 2^31
    for (int j = 0; j < 256; ++j) t.t[j] = (uint32_t)llroundl(ldexpl(exp2l(-(long double)j / 256.0L), 31));
    return t;
  }();
  return tab.t;
}

void launch_quantize(const float* z, int64_t n, uint16_t* freq, hipStream_t s) {
  if (n <= 0) return;
  QuantTab tab;
  const uint32_t* t = quant_table();
  for (int j = 0; j < 256; ++j) tab.t[j] = t[j];
  hipLaunchKernelGGL(k_quantize, dim3((unsigned)((n + 3) / 4)), dim3(256), 0, s, z, n, freq, tab);
}
