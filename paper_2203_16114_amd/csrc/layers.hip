// Stacked layers (Sec. 6.3, Fig. 7): the parts of the lower layers that are
// not matrix products.  A lower layer feeds every token of its output to the
// next layer, so unlike the top layer (attn.hip, ffn.hip: last query row
// only) its attention runs over all T query rows.  The projections, Wo and the
// FFN of these layers are GEMMs on the update's kernels (bgemm.hip, bwd.hip).
#include "kcommon.h"
#include "kernels.h"
#include "win.h"

// X[n][t][c] = E[byte j of group t of window n][c - j e] + P[t][c] (fp32, the
// sum of the operand copies): the tokens of Sec. 4.2 entering layer 0.
template <bool BF>
__global__ __launch_bounds__(256) void k_tokens(WinArgs w, const typename Mma<BF>::T* __restrict__ E,
                                                const typename Mma<BF>::T* __restrict__ P, int T, int D, int e, int g,
                                                float* __restrict__ X) {
  typedef Mma<BF> M;
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= w.N * T * D) return;
  const int c = (int)(i % D);
  const int64_t r = i / D;
  const int t = (int)(r % T);
  const int64_t n = r / T;
  const int j = c / e, cc = c - j * e;
  const int byte = w.streams[target_offset(w, n) - T * g + t * g + j];
  X[i] = M::val(E[byte * e + cc]) + M::val(P[t * D + c]);
}
void launch_tokens(bool bf, const WinArgs& w, const void* E, const void* P, int T, int D, int e, int g, float* X,
                   hipStream_t s) {
  const dim3 grid((unsigned)((w.N * T * D + 255) / 256));
  if (bf)
    hipLaunchKernelGGL(k_tokens<true>, grid, dim3(256), 0, s, w, (const uint16_t*)E, (const uint16_t*)P, T, D, e, g,
                       X);
  else
    hipLaunchKernelGGL(k_tokens<false>, grid, dim3(256), 0, s, w, (const float*)E, (const float*)P, T, D, e, g, X);
}

// Causal attention of Eqs. 1-2 over all T query rows of each (window, head):
// a wave (DH = 64) or half a wave (DH = 32) per pair, a lane per column.
// S[t][u] = scale Q[t].K[u] (shuffle sums over the head's lanes), u <= t;
// A = softmax over u; O[t] = sum_u A[t][u] V[u], written rounded to bf16
// when rb (the operand of Wo), and A kept when Akeep is not NULL.
template <int DH>
__global__ __launch_bounds__(256) void k_attn_rows(const float* __restrict__ Q, const float* __restrict__ K,
                                                   const float* __restrict__ V, int64_t N, int T, int D, int H,
                                                   float scale, int rb, float* __restrict__ O,
                                                   float* __restrict__ Akeep) {
  constexpr int PW = 64 / DH;
  const int lane = threadIdx.x & 63, c = lane % DH;
  const int64_t pair = ((int64_t)blockIdx.x * 4 + (threadIdx.x >> 6)) * PW + lane / DH;
  const int64_t np = N * H;
  const bool live = pair < np;
  const int64_t pr = live ? pair : 0;  // dead lanes redo pair 0 and store nothing
  const int64_t n = pr / H;
  const int h = (int)(pr % H);
  const int col = h * DH + c;
  float q[8], k[8], v[8];
#pragma unroll
  for (int t = 0; t < 8; ++t) {
    if (t < T) {
      q[t] = Q[(n * T + t) * D + col];
      k[t] = K[(n * T + t) * D + col];
      v[t] = V[(n * T + t) * D + col];
    }
  }
#pragma unroll
  for (int t = 0; t < 8; ++t) {
    if (t >= T) break;
    float sc[8];
    float mx = -__builtin_inff();
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      if (u <= t) {
        float x = q[t] * k[u];
#pragma unroll
        for (int off = 1; off < DH; off <<= 1) x += __shfl_xor(x, off, 64);
        sc[u] = x * scale;
        mx = fmaxf(mx, sc[u]);
      }
    }
    float tot = 0.f;
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      if (u <= t) {
        sc[u] = expf(sc[u] - mx);
        tot += sc[u];
      }
    }
    const float inv = 1.f / tot;
    float o = 0.f;
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      if (u < T) {
        const float a = u <= t ? sc[u] * inv : 0.f;
        o = fmaf(a, v[u], o);
        if (Akeep && live && c == 0) Akeep[((n * H + h) * T + t) * T + u] = a;
      }
    }
    if (live) O[(n * T + t) * D + col] = rb ? round_bf(o) : o;
  }
}
void launch_attn_rows(const float* Q, const float* K, const float* V, int64_t N, int T, int D, int H, float scale,
                      int rb, float* O, float* Akeep, hipStream_t s) {
  const int DH = D / H;
  const int64_t pairs = N * H, per_block = 4 * (64 / DH);
  const dim3 grid((unsigned)((pairs + per_block - 1) / per_block));
  if (DH == 32)
    hipLaunchKernelGGL(k_attn_rows<32>, grid, dim3(256), 0, s, Q, K, V, N, T, D, H, scale, rb, O, Akeep);
  else
    hipLaunchKernelGGL(k_attn_rows<64>, grid, dim3(256), 0, s, Q, K, V, N, T, D, H, scale, rb, O, Akeep);
}

// Its backward over all rows, same lanes: dA[t][u] = dO[t].V[u] (shuffle sums),
// dS[t][u] = A[t][u] (dA[t][u] - sum_u' A[t][u'] dA[t][u']); dQ[t] = scale
// sum_u dS[t][u] K[u], dK[u] = scale sum_t dS[t][u] Q[t], dV[u] = sum_t
// A[t][u] dO[t].  dO is the bf16 operand when rb.
template <int DH>
__global__ __launch_bounds__(256) void k_attn_bwd_rows(const float* __restrict__ dO, const float* __restrict__ Q,
                                                       const float* __restrict__ K, const float* __restrict__ V,
                                                       const float* __restrict__ A, int64_t N, int T, int D, int H,
                                                       float scale, int rb, float* __restrict__ dQ,
                                                       float* __restrict__ dK, float* __restrict__ dV) {
  const int lane = threadIdx.x & 63, c = lane % DH;
  const int64_t pair = ((int64_t)blockIdx.x * 4 + (threadIdx.x >> 6)) * (64 / DH) + lane / DH;
  const bool live = pair < N * H;
  const int64_t pr = live ? pair : 0;
  const int64_t n = pr / H;
  const int h = (int)(pr % H);
  const int col = h * DH + c;
  float q[8], k[8], v[8], o[8], dk[8], dv[8];
#pragma unroll
  for (int t = 0; t < 8; ++t) {
    dk[t] = dv[t] = 0.f;
    if (t < T) {
      q[t] = Q[(n * T + t) * D + col];
      k[t] = K[(n * T + t) * D + col];
      v[t] = V[(n * T + t) * D + col];
      const float x = dO[(n * T + t) * D + col];
      o[t] = rb ? round_bf(x) : x;
    }
  }
  const float* Ap = A + (n * H + h) * T * T;
#pragma unroll
  for (int t = 0; t < 8; ++t) {
    if (t >= T) break;
    float a[8], da[8];
    float tot = 0.f;
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      if (u <= t) {
        float x = o[t] * v[u];
#pragma unroll
        for (int off = 1; off < DH; off <<= 1) x += __shfl_xor(x, off, 64);
        da[u] = x;
        a[u] = Ap[t * T + u];
        tot = fmaf(a[u], x, tot);
      }
    }
    float dq = 0.f;
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      if (u <= t) {
        const float ds = a[u] * (da[u] - tot);
        dq = fmaf(ds, k[u], dq);
        dk[u] = fmaf(ds, q[t], dk[u]);
        dv[u] = fmaf(a[u], o[t], dv[u]);
      }
    }
    if (live) dQ[(n * T + t) * D + col] = dq * scale;
  }
  if (live) {
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      if (u < T) {
        dK[(n * T + u) * D + col] = dk[u] * scale;
        dV[(n * T + u) * D + col] = dv[u];
      }
    }
  }
}
void launch_attn_bwd_rows(const float* dO, const float* Q, const float* K, const float* V, const float* A, int64_t N,
                          int T, int D, int H, float scale, int rb, float* dQ, float* dK, float* dV, hipStream_t s) {
  const int DH = D / H;
  const int64_t pairs = N * H, per_block = 4 * (64 / DH);
  const dim3 grid((unsigned)((pairs + per_block - 1) / per_block));
  if (DH == 32)
    hipLaunchKernelGGL(k_attn_bwd_rows<32>, grid, dim3(256), 0, s, dO, Q, K, V, A, N, T, D, H, scale, rb, dQ, dK, dV);
  else
    hipLaunchKernelGGL(k_attn_bwd_rows<64>, grid, dim3(256), 0, s, dO, Q, K, V, A, N, T, D, H, scale, rb, dQ, dK, dV);
}
