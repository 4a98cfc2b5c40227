// Forward estimator of TRACE on gfx950: byte-grouping gather (Sec. 4.2), causal
// multi-head attention on the last token (Eqs. 1-2), the layer residuals of
// Eq. 4 with the FFN of Eq. 3 shared k times (Sec. 4.3), and the 256-way
// softmax head giving the code length -log2 p(next byte) (Alg. 2, line 3).
//
// Two fused kernels per chunk of windows:
//   k_attn      (this file) bytes -> tokens X (LDS) -> q (last token), K/V per
//               head (MFMA) -> softmax over the T keys -> O (LDS) -> O.Wo + X_last
//               = h0 (HBM)
//   k_ffn_head  (ffn.hip) h0 -> k x [h += GELU(h.W1).W2] with F streamed in
//               chunks, h kept in accumulator registers -> z = h.Wout + bout -> bits
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
// column nb*16 + l%16 and k = ks*KS + (l/16)*EPF + j, j < EPF.
template <bool BF>
__global__ void k_pack(const float* __restrict__ W, int K, int N, uint4* __restrict__ out) {
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
  for (int j = 0; j < M::EPF; ++j) v[j] = W[(int64_t)(kb + j) * N + n];
  union { uint4 u; typename M::T t[M::EPF]; } r;
#pragma unroll
  for (int j = 0; j < M::EPF; ++j) r.t[j] = M::cvt(v[j]);
  out[i] = r.u;
}

void launch_pack(bool bf, const float* W, int K, int N, void* out, hipStream_t s) {
  const int KS = bf ? 32 : 16;
  const int64_t total = (int64_t)(K / KS) * (N / 16) * 64;
  const dim3 grid((unsigned)((total + 255) / 256));
  if (bf)
    hipLaunchKernelGGL(k_pack<true>, grid, dim3(256), 0, s, W, K, N, (uint4*)out);
  else
    hipLaunchKernelGGL(k_pack<false>, grid, dim3(256), 0, s, W, K, N, (uint4*)out);
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
  const float x = M::val(E[byte * e + cc]) + M::val(P[t * D + c]);
  X[i] = M::val(M::cvt(x));
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

// ----------------------------------------------------------- attention block ----
// One workgroup (4 waves) per tile of MA windows = MA*T token rows.
//   * the tile's tokens X are built once in LDS (operand type);
//   * q = X_last.Wq (rows = the MA last tokens; waves split the D columns);
//   * wave w takes heads w, w+4, ...: [K_h | V_h] = X.[Wk_h | Wv_h] over all rows
//     stays in registers, and the softmax of the last row and O_h = a.V_h are
//     formed there with cross-lane reductions (a window's T rows sit in one or two
//     16-lane groups of the MFMA result);
//   * h0 = O.Wo + X_last (fp32 residual, Eq. 4).
// Only the last query row is needed: with one layer the head reads the last
// token, and under the causal mask row T-1 attends to every key.
template <bool BF, int T, int D, int DH, int MA>
__global__ __launch_bounds__(256) void k_attn(AttnArgs a) {
  typedef Mma<BF> M;
  typedef typename M::T OT;
  constexpr int H = D / DH;
  constexpr int ROWS = MA * T;
  constexpr int XSTR = D * (int)sizeof(OT) + 16;  // LDS row pitch in bytes (16 B pad)
  constexpr int KSTEPS = D / M::KS;
  constexpr int NB = D / 16;
  constexpr int RF = ROWS / 16;
  constexpr int NFH = DH / 16;
  constexpr int RFQ = (MA + 15) / 16;
  constexpr int NFQ = D / 64;
  static_assert(ROWS % 16 == 0 && D % 64 == 0 && DH % 16 == 0 && (T == 4 || T == 8), "shape");
  __shared__ __align__(16) unsigned char Xs[ROWS * XSTR];
  __shared__ __align__(16) unsigned char Os[RFQ * 16 * XSTR];
  __shared__ __align__(16) float Qs[MA * D];
  __shared__ uint8_t Wb[MA * 64];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, lg = lane >> 4, lc = lane & 15;
  const int64_t tile0 = (int64_t)blockIdx.x * MA;
  const int64_t N = a.w.N;
  const int W = T * a.g;
  const OT* __restrict__ E = (const OT*)a.E;
  const OT* __restrict__ P = (const OT*)a.P;

  // window bytes (tail windows of the last tile read nothing and are not stored)
  for (int i = tid; i < MA * W; i += 256) {
    const int m = i / W, j = i - m * W;
    const int64_t n = tile0 + m;
    uint8_t v = 0;
    if (n < N) {
      v = a.w.streams[target_offset(a.w, n) - W + j];
      if (a.kwin) a.kwin[n * W + j] = v;
    }
    Wb[m * 64 + j] = v;
  }
  __syncthreads();

  // byte-grouped tokens
  constexpr int CG = D / 8;
  for (int i = tid; i < ROWS * CG; i += 256) {
    const int r = i / CG, c8 = (i - r * CG) * 8;
    const int m = r / T, t = r - m * T;
    const int j = c8 / a.e, cc = c8 - j * a.e;
    const int byte = Wb[m * 64 + t * a.g + j];
    float ev[8], pv[8];
    load8(E + byte * a.e + cc, ev);
    load8(P + t * D + c8, pv);
#pragma unroll
    for (int q = 0; q < 8; ++q) ev[q] += pv[q];
    store8((OT*)(Xs + r * XSTR) + c8, ev);
  }
  __syncthreads();

  // q = X_last . Wq
  {
    f32x4 acc[RFQ][NFQ];
#pragma unroll
    for (int rf = 0; rf < RFQ; ++rf)
#pragma unroll
      for (int nf = 0; nf < NFQ; ++nf) acc[rf][nf] = f32x4{0.f, 0.f, 0.f, 0.f};
    const unsigned char* arow[RFQ];
#pragma unroll
    for (int rf = 0; rf < RFQ; ++rf) {
      int m = rf * 16 + lc;
      if (m >= MA) m = 0;
      arow[rf] = Xs + (m * T + T - 1) * XSTR + lg * 16;
    }
    for (int ks = 0; ks < KSTEPS; ++ks) {
      uint4 bq[NFQ];
#pragma unroll
      for (int nf = 0; nf < NFQ; ++nf) bq[nf] = a.Wq[(ks * NB + wave * NFQ + nf) * 64 + lane];
#pragma unroll
      for (int rf = 0; rf < RFQ; ++rf) {
        const uint4 af = *(const uint4*)(arow[rf] + ks * 64);
#pragma unroll
        for (int nf = 0; nf < NFQ; ++nf) M::run(acc[rf][nf], af, bq[nf]);
      }
    }
#pragma unroll
    for (int rf = 0; rf < RFQ; ++rf)
#pragma unroll
      for (int nf = 0; nf < NFQ; ++nf)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int m = rf * 16 + 4 * lg + r;
          const int col = (wave * NFQ + nf) * 16 + lc;
          if (m < MA) {
            Qs[m * D + col] = acc[rf][nf][r];
            if (a.kq && tile0 + m < N) a.kq[(tile0 + m) * D + col] = acc[rf][nf][r];
          }
        }
  }
  __syncthreads();

  // per head: K_h, V_h for all rows, then the last row's attention
  for (int h = wave; h < H; h += 4) {
    f32x4 acc[RF][2 * NFH];
#pragma unroll
    for (int rf = 0; rf < RF; ++rf)
#pragma unroll
      for (int nf = 0; nf < 2 * NFH; ++nf) acc[rf][nf] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int ks = 0; ks < KSTEPS; ++ks) {
      uint4 bk[NFH], bv[NFH];
#pragma unroll
      for (int nf = 0; nf < NFH; ++nf) {
        bk[nf] = a.Wk[(ks * NB + h * NFH + nf) * 64 + lane];
        bv[nf] = a.Wv[(ks * NB + h * NFH + nf) * 64 + lane];
      }
#pragma unroll
      for (int rf = 0; rf < RF; ++rf) {
        const uint4 af = *(const uint4*)(Xs + (rf * 16 + lc) * XSTR + ks * 64 + lg * 16);
#pragma unroll
        for (int nf = 0; nf < NFH; ++nf) {
          M::run(acc[rf][nf], af, bk[nf]);
          M::run(acc[rf][NFH + nf], af, bv[nf]);
        }
      }
    }
#pragma unroll
    for (int rf = 0; rf < RF; ++rf) {
      const int m = (T == 8) ? rf * 2 + (lg >> 1) : rf * 4 + lg;  // window of this lane's rows
      const int t0 = (T == 8) ? (lg & 1) * 4 : 0;                 // token of its first row
      float s[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int nf = 0; nf < NFH; ++nf) {
        const float qv = Qs[m * D + h * DH + nf * 16 + lc];
#pragma unroll
        for (int r = 0; r < 4; ++r) s[r] += qv * acc[rf][nf][r];
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) s[r] = wave_sum16(s[r]) * a.scale;
      float mx = fmaxf(fmaxf(s[0], s[1]), fmaxf(s[2], s[3]));
      if (T == 8) mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
      float p[4], sm = 0.f;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        p[r] = expf(s[r] - mx);
        sm += p[r];
      }
      if (T == 8) sm += __shfl_xor(sm, 16, 64);
#pragma unroll
      for (int r = 0; r < 4; ++r) p[r] = p[r] / sm;
      const int64_t n = tile0 + m;
      const bool keep = (n < N) && (m < MA);
#pragma unroll
      for (int nf = 0; nf < NFH; ++nf) {
        float o = 0.f;
#pragma unroll
        for (int r = 0; r < 4; ++r) o += p[r] * acc[rf][NFH + nf][r];
        if (T == 8) o += __shfl_xor(o, 16, 64);
        const int col = h * DH + nf * 16 + lc;
        if (T == 4 || (lg & 1) == 0) {
          const OT ov = M::cvt(o);
          ((OT*)(Os + m * XSTR))[col] = ov;
          if (a.kO && keep) a.kO[n * D + col] = M::val(ov);
        }
        if (a.kK && keep) {
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            a.kK[(n * T + t0 + r) * D + col] = acc[rf][nf][r];
            a.kV[(n * T + t0 + r) * D + col] = acc[rf][NFH + nf][r];
          }
        }
      }
      if (a.kA && keep && lc == 0) {
#pragma unroll
        for (int r = 0; r < 4; ++r) a.kA[(n * H + h) * T + t0 + r] = p[r];
      }
    }
  }
  __syncthreads();

  // h0 = O . Wo + X_last
  {
    f32x4 acc[RFQ][NFQ];
#pragma unroll
    for (int rf = 0; rf < RFQ; ++rf)
#pragma unroll
      for (int nf = 0; nf < NFQ; ++nf) acc[rf][nf] = f32x4{0.f, 0.f, 0.f, 0.f};
    const unsigned char* orow[RFQ];
#pragma unroll
    for (int rf = 0; rf < RFQ; ++rf) {
      int m = rf * 16 + lc;
      if (m >= MA) m = 0;
      orow[rf] = Os + m * XSTR + lg * 16;
    }
    for (int ks = 0; ks < KSTEPS; ++ks) {
      uint4 bo[NFQ];
#pragma unroll
      for (int nf = 0; nf < NFQ; ++nf) bo[nf] = a.Wo[(ks * NB + wave * NFQ + nf) * 64 + lane];
#pragma unroll
      for (int rf = 0; rf < RFQ; ++rf) {
        const uint4 af = *(const uint4*)(orow[rf] + ks * 64);
#pragma unroll
        for (int nf = 0; nf < NFQ; ++nf) M::run(acc[rf][nf], af, bo[nf]);
      }
    }
#pragma unroll
    for (int rf = 0; rf < RFQ; ++rf)
#pragma unroll
      for (int nf = 0; nf < NFQ; ++nf) {
        const int col = (wave * NFQ + nf) * 16 + lc;
        const int j = col / a.e, cc = col - j * a.e;
        const float pv = M::val(P[(T - 1) * D + col]);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int m = rf * 16 + 4 * lg + r;
          if (m < MA && tile0 + m < N) {
            const int byte = Wb[m * 64 + (T - 1) * a.g + j];
            const float x = M::val(E[byte * a.e + cc]) + pv;
            a.h0[(tile0 + m) * D + col] = acc[rf][nf][r] + x;
          }
        }
      }
  }
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

// ------------------------------------------------------------ dispatch ----
constexpr int attn_lds_bytes(bool bf, int T, int D, int ma) {
  return ma * T * (D * (bf ? 2 : 4) + 16) + ((ma + 15) / 16) * 16 * (D * (bf ? 2 : 4) + 16) + ma * D * 4 + ma * 64;
}
constexpr int pick_ma(bool bf, int T, int D, int DH) {
  int ma = 4096 / (T * DH);
  if (ma > 16) ma = 16;
  while (ma > 2 && attn_lds_bytes(bf, T, D, ma) > 160 * 1024) ma /= 2;
  return ma;
}
template <bool BF, int T, int D, int DH>
static void run_attn(const AttnArgs& a, hipStream_t s) {
  constexpr int MA = pick_ma(BF, T, D, DH);
  static_assert(attn_lds_bytes(BF, T, D, MA) <= 160 * 1024, "LDS");
  const dim3 grid((unsigned)((a.w.N + MA - 1) / MA));
  hipLaunchKernelGGL((k_attn<BF, T, D, DH, MA>), grid, dim3(256), 0, s, a);
}
attn_fn find_attn(bool bf, int T, int D, int DH) {
#define TRACE_ATTN(BF_, T_, D_, DH_) \
  if (bf == BF_ && T == T_ && D == D_ && DH == DH_) return &run_attn<BF_, T_, D_, DH_>;
#define TRACE_ATTN_T(BF_, D_, DH_) TRACE_ATTN(BF_, 4, D_, DH_) TRACE_ATTN(BF_, 8, D_, DH_)
  TRACE_ATTN_T(true, 64, 32) TRACE_ATTN_T(true, 64, 64) TRACE_ATTN_T(true, 128, 32) TRACE_ATTN_T(true, 128, 64)
  TRACE_ATTN_T(true, 256, 32) TRACE_ATTN_T(true, 256, 64) TRACE_ATTN_T(true, 512, 64)
  TRACE_ATTN_T(false, 64, 32) TRACE_ATTN_T(false, 64, 64) TRACE_ATTN_T(false, 128, 32) TRACE_ATTN_T(false, 128, 64)
  TRACE_ATTN_T(false, 256, 32) TRACE_ATTN_T(false, 256, 64)
#undef TRACE_ATTN_T
#undef TRACE_ATTN
  return nullptr;
}

