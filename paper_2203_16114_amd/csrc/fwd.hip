// Forward estimator of TRACE on gfx950: byte-grouping gather (Sec. 4.2), causal
// multi-head attention on the last token (Eqs. 1-2), the layer residuals of
// Eq. 4 with the FFN of Eq. 3 shared k times (Sec. 4.3), and the 256-way
// softmax head giving the code length -log2 p(next byte) (Alg. 2, line 3).
//
// Two fused kernels per chunk of windows:
//   k_attn      (attn.hip) bytes -> tokens X -> q (last token), K/V per head
//               (MFMA) -> softmax over the T keys -> O -> O.Wo + X_last = h0 (HBM)
//   k_ffn_head  (ffn.hip) h0 -> k x [h += GELU(h.W1).W2] with F streamed in
//               chunks, h kept in accumulator registers -> z = h.Wout + bout -> bits
// This file holds the small kernels around them: operand packing, the gather
// used by tests, and the per-step mean code length.
// Weights are read from L2 in a fragment-packed layout (see k_pack), one 16-byte
// load per lane per 16x16 fragment; activations stay in LDS or registers.  The
// only per-window HBM traffic is the window bytes, h0 (d floats written and read
// once) and the code length.
#include "kcommon.h"
#include "kernels.h"

#include "win.h"

// ------------------------------------------------------------------ packing ----
// W [K][N] row-major fp32 -> fragment-packed operand copy: fragment (ks, nb) is
// 64 lanes x 16 bytes at offset ((ks * N/16 + nb) * 64 + lane) * 16; lane l holds
// column nb*16 + l%16 and k = ks*KS + (l/16)*EPF + j, j < EPF.  Each value is
// multiplied by scale (a power of two, so the operand is the scaled rounded value).
template <bool BF>
__global__ void k_pack(const float* __restrict__ W, int K, int N, uint4* __restrict__ out, float scale) {
  typedef Mma<BF> M;
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int NB = N / 16, KSN = K / M::KS;
  if (i >= (int64_t)KSN * NB * 64) return;
  const int lane = (int)(i & 63);
  const int64_t f = i >> 6;
  const int nb = (int)(f % NB), ks = (int)(f / NB);
  const int n = nb * 16 + (lane & 15);
  const int kb = ks * M::KS + (lane >> 4) * M::EPF;
  float v[8];
#pragma unroll
  for (int j = 0; j < M::EPF; ++j) v[j] = W[(int64_t)(kb + j) * N + n] * scale;
  union { uint4 u; typename M::T t[M::EPF]; } r;
#pragma unroll
  for (int j = 0; j < M::EPF; ++j) r.t[j] = M::cvt(v[j]);
  out[i] = r.u;
}

void launch_pack(bool bf, const float* W, int K, int N, void* out, hipStream_t s, float scale) {
  const int KS = bf ? 32 : 16;
  const int64_t total = (int64_t)(K / KS) * (N / 16) * 64;
  const dim3 grid((unsigned)((total + 255) / 256));
  if (bf)
    hipLaunchKernelGGL(k_pack<true>, grid, dim3(256), 0, s, W, K, N, (uint4*)out, scale);
  else
    hipLaunchKernelGGL(k_pack<false>, grid, dim3(256), 0, s, W, K, N, (uint4*)out, scale);
}

// Positional parts of the projections: PW[w][t][j] = sum_i P[t][i] W_w[i][j] for
// w = q, k, v, in fp32 (eight partial sums over consecutive eighths of i, added in
// order), from the operand values of P
// and of the weights (bf16-rounded in BF16 mode).  A token's projection is then
// E-part (an MFMA on the rounded byte embeddings) + PW[w][t]: X.W = E.W + P.W.
template <bool BF>
__global__ __launch_bounds__(512) void k_ptab(const typename Mma<BF>::T* __restrict__ P, const float* __restrict__ Wq,
                                              const float* __restrict__ Wk, const float* __restrict__ Wv, int T, int D,
                                              float* __restrict__ PW) {
  // block (w*T + t, j-block): 64 columns j; its 8 waves sum over the 8 eighths of
  // k, and the 8 partial sums are added in k order
  typedef Mma<BF> M;
  __shared__ float part[8][64];
  const int wt = blockIdx.x, w = wt / T, t = wt - w * T;
  const int j = blockIdx.y * 64 + (threadIdx.x & 63), kg = threadIdx.x >> 6;
  const float* Wm = w == 0 ? Wq : (w == 1 ? Wk : Wv);
  const int kl = D / 8, k0 = kg * kl;
  float s = 0.f;
  if (j < D) {
#pragma unroll 4
    for (int k = k0; k < k0 + kl; ++k) s = fmaf(M::val(P[t * D + k]), M::val(M::cvt(Wm[(int64_t)k * D + j])), s);
  }
  part[kg][threadIdx.x & 63] = s;
  __syncthreads();
  if (kg == 0 && j < D) {
    float r = part[0][threadIdx.x];
#pragma unroll
    for (int q = 1; q < 8; ++q) r += part[q][threadIdx.x];
    PW[(int64_t)wt * D + j] = r;
  }
}

void launch_ptab(bool bf, const void* P, const float* Wq, const float* Wk, const float* Wv, int T, int D, float* PW,
                 hipStream_t s) {
  const dim3 grid((unsigned)(3 * T), (unsigned)((D + 63) / 64));
  if (bf)
    hipLaunchKernelGGL(k_ptab<true>, grid, dim3(512), 0, s, (const uint16_t*)P, Wq, Wk, Wv, T, D, PW);
  else
    hipLaunchKernelGGL(k_ptab<false>, grid, dim3(512), 0, s, (const float*)P, Wq, Wk, Wv, T, D, PW);
}

template <bool BF>
__global__ void k_cvt(const float* __restrict__ src, typename Mma<BF>::T* __restrict__ dst, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i < n) dst[i] = Mma<BF>::cvt(src[i]);
}
void launch_cvt(bool bf, const float* src, void* dst, int64_t n, hipStream_t s) {
  const dim3 grid((unsigned)((n + 255) / 256));
  if (bf)
    hipLaunchKernelGGL(k_cvt<true>, grid, dim3(256), 0, s, src, (uint16_t*)dst, n);
  else
    hipLaunchKernelGGL(k_cvt<false>, grid, dim3(256), 0, s, src, (float*)dst, n);
}

__global__ void k_zero(uint32_t* __restrict__ p, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i < n) p[i] = 0u;
}
// Clears n32 32-bit words with a kernel (not a memset node, so it is safe under
// graph capture).
void launch_zero(void* p, int64_t n32, hipStream_t s) {
  if (n32 > 0) hipLaunchKernelGGL(k_zero, dim3((unsigned)((n32 + 255) / 256)), dim3(256), 0, s, (uint32_t*)p, n32);
}

// ------------------------------------------------------------ gather (debug) ----
// Token operand values X[n][t][c] of Sec. 4.2: byte j of group t (oldest first)
// fills columns [j*e, (j+1)*e) with E[byte]; P[t] is added in fp32, then the sum
// is rounded to the operand type.
template <bool BF>
__global__ void k_gather(WinArgs w, const typename Mma<BF>::T* __restrict__ E, const typename Mma<BF>::T* __restrict__ P,
                         int T, int D, int e, int g, float* __restrict__ X) {
  typedef Mma<BF> M;
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t total = w.N * T * D;
  if (i >= total) return;
  const int c = (int)(i % D);
  const int64_t r = i / D;
  const int t = (int)(r % T);
  const int64_t n = r / T;
  const int j = c / e, cc = c - j * e;
  const int W = T * g;
  const int byte = w.streams[target_offset(w, n) - W + t * g + j];
  X[i] = M::val(E[byte * e + cc]) + M::val(P[t * D + c]);
}
void launch_gather(bool bf, const WinArgs& w, const void* E, const void* P, int T, int D, int e, int g, float* X,
                   hipStream_t s) {
  const int64_t total = w.N * T * D;
  const dim3 grid((unsigned)((total + 255) / 256));
  if (bf)
    hipLaunchKernelGGL(k_gather<true>, grid, dim3(256), 0, s, w, (const uint16_t*)E, (const uint16_t*)P, T, D, e, g,
                       X);
  else
    hipLaunchKernelGGL(k_gather<false>, grid, dim3(256), 0, s, w, (const float*)E, (const float*)P, T, D, e, g, X);
}

// ------------------------------------------------------------- step means ----
// step_ce[s] = (1/B) sum_b bits[b][s] in double, in a fixed order.
__global__ __launch_bounds__(256) void k_step_ce(const float* __restrict__ bits, int32_t n_streams, int32_t n_steps,
                                                 double* __restrict__ out) {
  __shared__ double sh[256];
  const int s = blockIdx.x, tid = threadIdx.x;
  double acc = 0.0;
  for (int b = tid; b < n_streams; b += 256) acc += (double)bits[(int64_t)b * n_steps + s];
  sh[tid] = acc;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (tid < w) sh[tid] += sh[tid + w];
    __syncthreads();
  }
  if (tid == 0) out[s] = sh[0] / (double)n_streams;
}
void launch_step_ce(const float* bits, int32_t n_streams, int32_t n_steps, double* out, hipStream_t s) {
  hipLaunchKernelGGL(k_step_ce, dim3(n_steps), dim3(256), 0, s, bits, n_streams, n_steps, out);
}

