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
// Weights are read from L2 in a fragment-packed layout (see refresh_pack), one 16-byte
// load per lane per 16x16 fragment; activations stay in LDS or registers.  The
// only per-window HBM traffic is the window bytes, h0 (d floats written and read
// once) and the code length.
#include "kcommon.h"
#include "kernels.h"

#include "win.h"

// ------------------------------------------------------------------ refresh ----
// Every operand copy of the model is derived from the fp32 master in one launch:
// each job (kernels.h) owns a consecutive range of blocks, and a block finds its
// job by comparing its index with the ranges' starts.
struct RefreshArgs {
  RefreshJob job[REFRESH_MAX_JOBS];
  int b0[REFRESH_MAX_JOBS + 1];  // first block of each job; b0[n] = grid size
  int n;
};

// Fragment-packed operand copy: fragment (ks, nb) of W [K][N] is 64 lanes x 16
// bytes at offset ((ks * N/16 + nb) * 64 + lane) * 16; lane l holds column
// nb*16 + l%16 and k = ks*KS + (l/16)*EPF + j, j < EPF.  Each value is multiplied
// by scale (a power of two, so the operand is the scaled rounded value).
template <bool BF>
__device__ __forceinline__ void refresh_pack(const RefreshJob& jb, int64_t i) {
  typedef Mma<BF> M;
  const int NB = jb.N / 16, KSN = jb.K / M::KS;
  if (i >= (int64_t)KSN * NB * 64) return;
  const int lane = (int)(i & 63);
  const int64_t f = i >> 6;
  const int nb = (int)(f % NB), ks = (int)(f / NB);
  const int n = nb * 16 + (lane & 15);
  const int kb = ks * M::KS + (lane >> 4) * M::EPF;
  float v[8];
  if (jb.kind == RJ_PACKT) {  // src is [N][K]: element (k, n) of its transpose at src[n * K + k]
    // (16-byte aligned: launch_refresh checks src and K)
#pragma unroll
    for (int j = 0; j < M::EPF; j += 4) {
      const float4 x = *reinterpret_cast<const float4*>(jb.src + (int64_t)n * jb.K + kb + j);
      v[j] = x.x * jb.scale;
      v[j + 1] = x.y * jb.scale;
      v[j + 2] = x.z * jb.scale;
      v[j + 3] = x.w * jb.scale;
    }
  } else {
#pragma unroll
    for (int j = 0; j < M::EPF; ++j) v[j] = jb.src[(int64_t)(kb + j) * jb.N + n] * jb.scale;
  }
  union { uint4 u; typename M::T t[M::EPF]; } r;
#pragma unroll
  for (int j = 0; j < M::EPF; ++j) r.t[j] = M::cvt(v[j]);
  reinterpret_cast<uint4*>(jb.dst)[i] = r.u;
}

// Positional parts of the projections, PW[w][t][j] = sum_i P[t][i] W_w[i][j]
// (w = q, k, v), in fp32 from the operand values of P and of the weights, so that
// a token's projection is an MFMA on the rounded byte embeddings plus PW[w][t]:
// X.W = E.W + P.W.  A block takes 16 columns j of one W_w for every token t; its
// 16 thread groups of 16 take consecutive sixteenths of i, read each weight value
// once for all tokens, and their 16 partial sums are added in i order.  A thread
// issues all of its weight loads (at most 32) before it stages P, so that one
// memory latency covers them.
constexpr int PTAB_TMAX = 8, PTAB_DMAX = 512;
template <bool BF, int T>
__device__ __forceinline__ void refresh_ptab(const RefreshJob& jb, int lb, float* Pv, float* part) {
  typedef Mma<BF> M;
  constexpr int KLMAX = PTAB_DMAX / 16;
  const int D = jb.N, nbw = D / 16;
  const int w = lb / nbw, j = (lb - w * nbw) * 16 + (threadIdx.x & 15), kg = threadIdx.x >> 4;
  const float* Wm = jb.src2 + (int64_t)w * D * D + j;
  const int kl = D / 16, k0 = kg * kl;  // kl is a multiple of 4 (D a multiple of 64)
  float wv[KLMAX];
#pragma unroll
  for (int u = 0; u < KLMAX; ++u) wv[u] = Wm[(int64_t)(k0 + min(u, kl - 1)) * D];  // (clamped: u < kl used)
  {  // every load of P first (float4; T D is a multiple of 4, src 16-byte aligned)
    constexpr int NU = PTAB_TMAX * PTAB_DMAX / 4 / 256;
    const int n4 = T * D / 4;
    float4 x[NU];
#pragma unroll
    for (int u = 0; u < NU; ++u) {
      const int i = threadIdx.x + 256 * u;
      x[u] = (jb.use_pos && i < n4) ? reinterpret_cast<const float4*>(jb.src)[i] : make_float4(0.f, 0.f, 0.f, 0.f);
    }
#pragma unroll
    for (int u = 0; u < NU; ++u) {
      const int i = threadIdx.x + 256 * u;
      if (i < n4)
        reinterpret_cast<float4*>(Pv)[i] = make_float4(M::val(M::cvt(x[u].x)), M::val(M::cvt(x[u].y)),
                                                       M::val(M::cvt(x[u].z)), M::val(M::cvt(x[u].w)));
    }
  }
  __syncthreads();
  float acc[T];
#pragma unroll
  for (int t = 0; t < T; ++t) acc[t] = 0.f;
#pragma unroll
  for (int u = 0; u < KLMAX; u += 4) {
    if (u < kl) {
      float x[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) x[e] = M::val(M::cvt(wv[u + e]));
#pragma unroll
      for (int t = 0; t < T; ++t) {
        const float4 p = *reinterpret_cast<const float4*>(Pv + t * D + k0 + u);
        acc[t] = fmaf(p.x, x[0], acc[t]);
        acc[t] = fmaf(p.y, x[1], acc[t]);
        acc[t] = fmaf(p.z, x[2], acc[t]);
        acc[t] = fmaf(p.w, x[3], acc[t]);
      }
    }
  }
  __syncthreads();  // (part overlays Pv)
#pragma unroll
  for (int t = 0; t < T; ++t) part[(kg * T + t) * 16 + (threadIdx.x & 15)] = acc[t];
  __syncthreads();
  if ((int)threadIdx.x < T * 16) {
    const int t = threadIdx.x >> 4, c = threadIdx.x & 15;
    float r = part[t * 16 + c];
#pragma unroll
    for (int q = 1; q < 16; ++q) r += part[(q * T + t) * 16 + c];
    reinterpret_cast<float*>(jb.dst)[(int64_t)(w * T + t) * D + (lb - w * nbw) * 16 + c] = r;
  }
}

// (16 KB of LDS per block, the partial sums over the staged P: every block of a
// launch of about 2000 can be resident at once)
template <bool BF>
__global__ __launch_bounds__(256) void k_refresh(RefreshArgs a) {
  static_assert(16 * PTAB_TMAX * 16 <= PTAB_TMAX * PTAB_DMAX, "part fits in Pv");
  __shared__ __align__(16) float Pv[PTAB_TMAX * PTAB_DMAX];
  float* const part = Pv;
  const int b = (int)blockIdx.x;
  int q = 0;
#pragma unroll
  for (int u = 1; u < REFRESH_MAX_JOBS; ++u) q += (u < a.n && b >= a.b0[u]) ? 1 : 0;
  // the job's fields, selected with constant indexes (the block index is uniform)
  RefreshJob jb = a.job[0];
  int b0 = a.b0[0];
#pragma unroll
  for (int u = 1; u < REFRESH_MAX_JOBS; ++u)
    if (q == u) {
      jb = a.job[u];
      b0 = a.b0[u];
    }
  const int lb = b - b0;
  const int64_t i = (int64_t)lb * 256 + threadIdx.x;
  typedef Mma<BF> M;
  if (jb.kind == RJ_CVT) {
    if (i < jb.K) reinterpret_cast<typename M::T*>(jb.dst)[i] = M::cvt(jb.src[i]);
  } else if (jb.kind == RJ_CVT8) {
    if (i < jb.K / 8) {
      const float4 x = reinterpret_cast<const float4*>(jb.src)[2 * i];
      const float4 y = reinterpret_cast<const float4*>(jb.src)[2 * i + 1];
      const float v[8] = {x.x, x.y, x.z, x.w, y.x, y.y, y.z, y.w};
      union { uint4 u; typename M::T t[8]; } r;
      static_assert(BF ? sizeof(r.t) == 16 : true, "eight bf16 values per 16 bytes");
      if constexpr (BF) {
#pragma unroll
        for (int j = 0; j < 8; ++j) r.t[j] = M::cvt(v[j]);
        reinterpret_cast<uint4*>(jb.dst)[i] = r.u;
      } else {
        reinterpret_cast<float4*>(jb.dst)[2 * i] = x;
        reinterpret_cast<float4*>(jb.dst)[2 * i + 1] = y;
      }
    }
  } else if (jb.kind == RJ_PACK || jb.kind == RJ_PACKT) {
    refresh_pack<BF>(jb, i);
  } else if (jb.kind == RJ_PTAB) {
    if (jb.K == 8)
      refresh_ptab<BF, 8>(jb, lb, Pv, part);
    else
      refresh_ptab<BF, 4>(jb, lb, Pv, part);
  } else {
    if (i < jb.K) reinterpret_cast<uint32_t*>(jb.dst)[i] = 0u;
  }
}

bool launch_refresh(bool bf, const RefreshJob* jobs, int n, hipStream_t s) {
  if (n < 1 || n > REFRESH_MAX_JOBS) return false;
  RefreshArgs a;
  int b = 0;
  for (int u = 0; u < n; ++u) {
    const RefreshJob& jb = jobs[u];
    int64_t nb = 0;
    if (jb.kind == RJ_CVT || jb.kind == RJ_ZERO) {
      nb = ((int64_t)jb.K + 255) / 256;
    } else if (jb.kind == RJ_CVT8) {
      if (jb.K % 8 != 0 || ((uintptr_t)jb.src & 15) != 0 || ((uintptr_t)jb.dst & 15) != 0) return false;
      nb = ((int64_t)jb.K / 8 + 255) / 256;
    } else if (jb.kind == RJ_PACK || jb.kind == RJ_PACKT) {
      const int KS = bf ? 32 : 16;
      if (jb.K % KS != 0 || jb.N % 16 != 0) return false;
      if (jb.kind == RJ_PACKT && ((uintptr_t)jb.src & 15) != 0) return false;
      nb = ((int64_t)(jb.K / KS) * (jb.N / 16) * 64 + 255) / 256;
    } else if (jb.kind == RJ_PTAB) {
      if ((jb.K != 4 && jb.K != 8) || jb.N > PTAB_DMAX || jb.N % 64 != 0) return false;
      if (jb.use_pos && ((uintptr_t)jb.src & 15) != 0) return false;
      nb = 3 * (int64_t)(jb.N / 16);
    } else {
      return false;
    }
    if (jb.K < 0 || b + nb > (1 << 30)) return false;
    a.job[u] = jb;
    a.b0[u] = b;
    b += (int)nb;
  }
  for (int u = n; u < REFRESH_MAX_JOBS; ++u) {
    a.job[u] = jobs[0];
    a.b0[u] = b;
  }
  a.b0[REFRESH_MAX_JOBS] = b;
  a.n = n;
  if (b == 0) return true;
  if (bf)
    hipLaunchKernelGGL(k_refresh<true>, dim3((unsigned)b), dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL(k_refresh<false>, dim3((unsigned)b), dim3(256), 0, s, a);
  return true;
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

