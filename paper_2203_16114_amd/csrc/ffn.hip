// Shared FFN applied k times and the 256-way softmax head, fused (Eq. 3, the
// layer of Eq. 4 with the FFN shared across repeats as in Sec. 4.3, and the
// code length -log2 p of Alg. 2, line 3).
//
// One workgroup of 8 waves per tile of MB windows.  Every product is formed
// transposed, weights as the MFMA A operand and windows as the B operand, so a
// lane's four results are four consecutive features of one window:
//   U^T = W1^T . Y^T    (chunk of FC features)       -> GELU -> G (LDS, [m][f])
//   Y^T += W2^T . G^T   (accumulators = residual)     -> bf(Y) (LDS, [m][d])
//   z^T = Wout^T . Y^T + bout                         -> log-sum-exp -> bits
// Waves form a 4 x 2 grid: 4 groups of output features x 2 groups of windows.
// The residual stream Y stays in accumulator registers for all k repeats; the
// weights stream from L2 in the fragment-packed layout, one k-step ahead of the
// MFMAs that use them; the activations are read from LDS.  k_ffn_head is the
// plain form (fp32 operands); k_ffn_pipe, further down, is the bf16 form, which
// overlaps the GELU with the MFMAs of neighbouring chunks.
#include <type_traits>

#include "kcommon.h"
#include "kernels.h"
#include "win.h"

// four fp32 values -> four operand elements at p (8 or 16 bytes)
__device__ __forceinline__ void put4(uint16_t* p, const f32x4& v) {
  *reinterpret_cast<uint2*>(p) = make_uint2(pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]));
}
__device__ __forceinline__ void put4(float* p, const f32x4& v) {
  *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
}

// Swizzled rows (a power of two of 16-byte units, no padding): unit u of row
// m is stored at unit u ^ (m & mask), mask = min(units, 16) - 1, which makes
// the 16-row fragment reads of the MFMA loops free of LDS bank conflicts.  A
// lane reads row m0 + lc (m0 a multiple of 16, so m & mask = lc & mask) at
// units 4 ks + lg, i.e. at byte 64 (ks & ~3) + off[ks & 3] of the row:
__device__ __forceinline__ void swz_off(int lg, int lc, int mask, int (&off)[4]) {
  const int q = (lc & mask) >> 2, p = lg ^ (lc & 3);
#pragma unroll
  for (int j = 0; j < 4; ++j) off[j] = 16 * (((j ^ q) << 2) | p);
}
// byte offset in a swizzled row of the 8-byte group holding elements e .. e+3
// (bf16, e a multiple of 4) of row m
__device__ __forceinline__ int swz_elem(int m, int e, int mask) { return 16 * ((e >> 3) ^ (m & mask)) + 8 * ((e >> 2) & 1); }

// Head on bf(Y_k) staged in Ys, then the code length (shared by both FFN
// kernels): z^T = Wout^T . Y^T + bout, log-sum-exp across the 4 feature waves
// through LDS in a fixed order, bits = log2 sum exp(z - max) - (z_y - max) log2 e
// (each exp(z - max) as the hardware 2^x of (z - max) log2 e: relative error
// about 1e-7 per term, against 1e-4 bits of parity tolerance).
// YM >= 0: Ys rows are unpadded and swizzled (unit u of row m at u ^ (m & YM),
// see swz_off); YM < 0: padded rows, unit u at u.
template <bool BF, int D, int MB, bool KEEP, int YSTR, int YM = -1>
__device__ __forceinline__ void ffn_head_out(const FfnArgs& a, const unsigned char* Ys, float (&red)[2][4][MB],
                                             float* zy, const int* tg) {
  typedef Mma<BF> M;
  typedef typename M::T OT;
  constexpr int WR = 4, WC = 2;
  constexpr int CW = MB / WC, NFC = CW / 16;
  constexpr int RFH = 256 / (WR * 16);
  constexpr int KD = D / M::KS;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, lg = lane >> 4, lc = lane & 15;
  const int wr = wave % WR, wc = wave / WR;
  const int64_t tile0 = (int64_t)blockIdx.x * MB;
  const int64_t N = a.w.N;
  const int m0 = wc * CW;
  const unsigned char* yrow[NFC];
#pragma unroll
  for (int nf = 0; nf < NFC; ++nf) yrow[nf] = Ys + (m0 + nf * 16 + lc) * YSTR + (YM < 0 ? lg * 16 : 0);
  int yo[4];
  if constexpr (YM >= 0) swz_off(lg, lc, YM, yo);
  f32x4 z[RFH][NFC];
#pragma unroll
  for (int rf = 0; rf < RFH; ++rf)
#pragma unroll
    for (int nf = 0; nf < NFC; ++nf) z[rf][nf] = f32x4{0.f, 0.f, 0.f, 0.f};
  uint4 wz[2][RFH];
#pragma unroll
  for (int rf = 0; rf < RFH; ++rf) wz[0][rf] = a.Wout[(wr * RFH + rf) * 64 + lane];
#pragma unroll
  for (int ks = 0; ks < KD; ++ks) {
    if (ks + 1 < KD) {
#pragma unroll
      for (int rf = 0; rf < RFH; ++rf) wz[(ks + 1) & 1][rf] = a.Wout[((ks + 1) * 16 + wr * RFH + rf) * 64 + lane];
    }
    uint4 bb[NFC];
#pragma unroll
    for (int nf = 0; nf < NFC; ++nf) {
      if constexpr (YM >= 0)
        bb[nf] = *(const uint4*)(yrow[nf] + (ks & ~3) * 64 + yo[ks & 3]);
      else
        bb[nf] = *(const uint4*)(yrow[nf] + ks * 64);
    }
#pragma unroll
    for (int rf = 0; rf < RFH; ++rf)
#pragma unroll
      for (int nf = 0; nf < NFC; ++nf) M::run(z[rf][nf], wz[ks & 1][rf], bb[nf]);
  }
  // lane holds z[v = wr*64 + rf*16 + 4*lg + r] of window m0 + nf*16 + lc
#pragma unroll
  for (int rf = 0; rf < RFH; ++rf) {
    const float4 bo = *reinterpret_cast<const float4*>(a.bout + wr * 64 + rf * 16 + 4 * lg);
#pragma unroll
    for (int nf = 0; nf < NFC; ++nf) {
      z[rf][nf][0] += bo.x;
      z[rf][nf][1] += bo.y;
      z[rf][nf][2] += bo.z;
      z[rf][nf][3] += bo.w;
    }
  }
#pragma unroll
  for (int nf = 0; nf < NFC; ++nf) {
    const int m = m0 + nf * 16 + lc;
    float mx = z[0][nf][0];
#pragma unroll
    for (int rf = 0; rf < RFH; ++rf)
#pragma unroll
      for (int r = 0; r < 4; ++r) mx = fmaxf(mx, z[rf][nf][r]);
    mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    if (lg == 0) red[0][wr][m] = mx;
    const int t = tg[m];
#pragma unroll
    for (int rf = 0; rf < RFH; ++rf)
#pragma unroll
      for (int r = 0; r < 4; ++r)
        if (wr * 64 + rf * 16 + 4 * lg + r == t) zy[m] = z[rf][nf][r];
  }
  __syncthreads();
#pragma unroll
  for (int nf = 0; nf < NFC; ++nf) {
    const int m = m0 + nf * 16 + lc;
    const int64_t n = tile0 + m;
    const float mx = fmaxf(fmaxf(red[0][0][m], red[0][1][m]), fmaxf(red[0][2][m], red[0][3][m]));
    const float mxl = -mx * TRACE_LOG2E;
    float se = 0.f;
#pragma unroll
    for (int rf = 0; rf < RFH; ++rf)
#pragma unroll
      for (int r = 0; r < 4; ++r) se += __builtin_amdgcn_exp2f(fmaf(z[rf][nf][r], TRACE_LOG2E, mxl));
    se += __shfl_xor(se, 16, 64);
    se += __shfl_xor(se, 32, 64);
    if (lg == 0) red[1][wr][m] = se;
    if (n < N) {
#pragma unroll
      for (int rf = 0; rf < RFH; ++rf) {
        const int v = wr * 64 + rf * 16 + 4 * lg;
        const float4 zz = make_float4(z[rf][nf][0], z[rf][nf][1], z[rf][nf][2], z[rf][nf][3]);
        if (a.logits) *reinterpret_cast<float4*>(a.logits + (a.w.n0 + n) * 256 + v) = zz;
        if (KEEP) *reinterpret_cast<float4*>(a.kZ + n * 256 + v) = zz;
      }
    }
  }
  __syncthreads();
  if (tid < MB) {
    const int m = tid;
    const int64_t n = tile0 + m;
    if (n < N) {
      const float mx = fmaxf(fmaxf(red[0][0][m], red[0][1][m]), fmaxf(red[0][2][m], red[0][3][m]));
      const float tot = ((red[1][0][m] + red[1][1][m]) + red[1][2][m]) + red[1][3][m];
      a.bits[a.w.n0 + n] = log2f(tot) - (zy[m] - mx) * TRACE_LOG2E;
    }
  }
}

template <bool BF, int D, int MB, int FC, bool KEEP>
__global__ __launch_bounds__(512) void k_ffn_head(FfnArgs a) {
  typedef Mma<BF> M;
  typedef typename M::T OT;
  constexpr int WR = 4, WC = 2;
  constexpr int CW = MB / WC, NFC = CW / 16;
  constexpr int RF1 = FC / (WR * 16), RF2 = D / (WR * 16), RFH = 256 / (WR * 16);
  constexpr int YSTR = D * (int)sizeof(OT) + 16, GSTR = FC * (int)sizeof(OT) + 16;
  constexpr int KD = D / M::KS, KC = FC / M::KS;
  constexpr int NB2 = D / 16;
  static_assert(RF1 >= 1 && RF2 >= 1 && NFC >= 1 && MB % (16 * WC) == 0, "shape");
  __shared__ __align__(16) unsigned char Ys[MB * YSTR];
  __shared__ __align__(16) unsigned char Gs[MB * GSTR];
  __shared__ float red[2][WR][MB];
  __shared__ float zy[MB];
  __shared__ int tg[MB];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, lg = lane >> 4, lc = lane & 15;
  const int wr = wave % WR, wc = wave / WR;
  const int64_t tile0 = (int64_t)blockIdx.x * MB;
  const int64_t N = a.w.N;
  const int F = a.F;
  const int NB1 = F / 16;
  const int d0 = wr * (D / WR);  // first feature row of this wave in Y / GEMM2
  const int f0 = wr * (FC / WR); // first feature row of this wave within a chunk
  const int m0 = wc * CW;        // first window (column) of this wave
  const uint4* W1p = a.W1;  // this repeat's W1, W2 (untied: advanced by wstride per repeat)
  const uint4* W2p = a.W2;

  // Y^T: lane holds Y[m0 + nf*16 + lc][d0 + rf*16 + 4*lg + r]
  f32x4 y[RF2][NFC];
#pragma unroll
  for (int nf = 0; nf < NFC; ++nf) {
    const int64_t n = tile0 + m0 + nf * 16 + lc;
#pragma unroll
    for (int rf = 0; rf < RF2; ++rf) {
      if (n < N) {
        const float4 v = *reinterpret_cast<const float4*>(a.h0 + n * D + d0 + rf * 16 + 4 * lg);
        y[rf][nf] = f32x4{v.x, v.y, v.z, v.w};
      } else {
        y[rf][nf] = f32x4{0.f, 0.f, 0.f, 0.f};
      }
    }
  }
  if (tid < MB) {
    const int64_t n = tile0 + tid;
    int v = 0;
    if (n < N) {
      v = a.w.streams[target_offset(a.w, n)];
      if (KEEP) a.ktgt[n] = v;
    }
    tg[tid] = v;
  }
  const unsigned char* yrow[NFC];
  const unsigned char* grow[NFC];
#pragma unroll
  for (int nf = 0; nf < NFC; ++nf) {
    yrow[nf] = Ys + (m0 + nf * 16 + lc) * YSTR + lg * 16;
    grow[nf] = Gs + (m0 + nf * 16 + lc) * GSTR + lg * 16;
  }

  uint4 wa[2][RF1];  // W1 fragments, double-buffered over k-steps
  uint4 wb[2][RF2];  // W2 fragments
#pragma unroll
  for (int rf = 0; rf < RF1; ++rf) wa[0][rf] = W1p[(f0 / 16 + rf) * 64 + lane];

  for (int rep = 0; rep <= a.k; ++rep) {
    if (rep > 0 && rep < a.k) {
      W1p += a.wstride;
      W2p += a.wstride;
    }
#pragma unroll
    for (int nf = 0; nf < NFC; ++nf) {
      const int m = m0 + nf * 16 + lc;
      const int64_t n = tile0 + m;
#pragma unroll
      for (int rf = 0; rf < RF2; ++rf) {
        const int dd = d0 + rf * 16 + 4 * lg;
        if (KEEP && n < N) put4((OT*)a.kY + ((int64_t)rep * N + n) * D + dd, y[rf][nf]);
        put4((OT*)(Ys + m * YSTR) + dd, y[rf][nf]);
      }
    }
    __syncthreads();
    if (rep == a.k) break;
    for (int c0 = 0; c0 < F; c0 += FC) {
      const int nb1 = (c0 + f0) / 16;
      f32x4 u[RF1][NFC];
#pragma unroll
      for (int rf = 0; rf < RF1; ++rf)
#pragma unroll
        for (int nf = 0; nf < NFC; ++nf) u[rf][nf] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < KD; ++ks) {
        if (ks + 1 < KD) {
#pragma unroll
          for (int rf = 0; rf < RF1; ++rf) wa[(ks + 1) & 1][rf] = W1p[((ks + 1) * NB1 + nb1 + rf) * 64 + lane];
        } else {
#pragma unroll
          for (int rf = 0; rf < RF2; ++rf) wb[0][rf] = W2p[((c0 / M::KS) * NB2 + d0 / 16 + rf) * 64 + lane];
        }
        uint4 bb[NFC];
#pragma unroll
        for (int nf = 0; nf < NFC; ++nf) bb[nf] = *(const uint4*)(yrow[nf] + ks * 64);
#pragma unroll
        for (int rf = 0; rf < RF1; ++rf)
#pragma unroll
          for (int nf = 0; nf < NFC; ++nf) M::run(u[rf][nf], wa[ks & 1][rf], bb[nf]);
      }
      // GELU of U^T into G[m][f] (four consecutive features per lane)
#pragma unroll
      for (int nf = 0; nf < NFC; ++nf) {
        const int m = m0 + nf * 16 + lc;
        const int64_t n = tile0 + m;
#pragma unroll
        for (int rf = 0; rf < RF1; ++rf) {
          const int fl = f0 + rf * 16 + 4 * lg;
          if (KEEP && n < N)
            *reinterpret_cast<float4*>(a.kU + ((int64_t)rep * N + n) * F + c0 + fl) =
                make_float4(u[rf][nf][0], u[rf][nf][1], u[rf][nf][2], u[rf][nf][3]);
          f32x4 gv;
#pragma unroll
          for (int r = 0; r < 4; ++r) gv[r] = gelu_as(u[rf][nf][r]);
          put4((OT*)(Gs + m * GSTR) + fl, gv);
        }
      }
      __syncthreads();
      const int kc0 = c0 / M::KS;
      const int nb1n = (((c0 + FC) % F) + f0) / 16;
#pragma unroll
      for (int ks = 0; ks < KC; ++ks) {
        if (ks + 1 < KC) {
#pragma unroll
          for (int rf = 0; rf < RF2; ++rf) wb[(ks + 1) & 1][rf] = W2p[((kc0 + ks + 1) * NB2 + d0 / 16 + rf) * 64 + lane];
        } else {
#pragma unroll
          for (int rf = 0; rf < RF1; ++rf)
            wa[0][rf] = (c0 + FC >= F && rep + 1 < a.k ? W1p + a.wstride : W1p)[(nb1n + rf) * 64 + lane];
        }
        uint4 bb[NFC];
#pragma unroll
        for (int nf = 0; nf < NFC; ++nf) bb[nf] = *(const uint4*)(grow[nf] + ks * 64);
#pragma unroll
        for (int rf = 0; rf < RF2; ++rf)
#pragma unroll
          for (int nf = 0; nf < NFC; ++nf) M::run(y[rf][nf], wb[ks & 1][rf], bb[nf]);
      }
      __syncthreads();
    }
  }

  ffn_head_out<BF, D, MB, KEEP, YSTR>(a, Ys, red, zy, tg);
}

// ------------------------------------------------- pipelined bf16 variant ----
// Same arithmetic as k_ffn_head (bf16 operands, fp32 accumulation, U rounded
// to bf16 after GELU; the GELU by the exp2 form gelu2_ex), restructured so that
// the GELU's vector ALU work runs in the same wave as independent MFMAs.  F is cut into chunks of 128 features
// and each interval between two barriers does, per wave:
//   GEMM2 of chunk j-1 (reads G from LDS buffer (j-1)&1, accumulates Y),
//   GEMM1 of chunk j+1 (reads bf(Y) from LDS, accumulates U into one register set),
//   GELU of chunk j    (the other register set, in place, written to buffer j&1),
// with one GELU value issued after every few MFMAs (scheduled as at most three
// vector instructions after each MFMA: a 16-cycle MFMA hides up to about three,
// more serialise).  The two U register sets
// alternate roles from one interval to the next; the loop takes two intervals
// per trip so that the roles stay compile-time.  G holds bf(2 GELU(U)) and the
// packed W2 copy holds bf(W2)/2: both scalings are exact, so every product is
// the one of bf(GELU(U)) and bf(W2), with one vector operation less per value.
template <int D, int MB, int WC_ = 2>
struct FfnPipe {
  // 8 waves: WR along features (GEMM1) / model dims (GEMM2), WC along windows
  static constexpr int FC = 128, WC = WC_, WR = 8 / WC_;
  static constexpr int CW = MB / WC, NFC = CW / 16;
  static constexpr int RF1 = FC / (WR * 16), RF2 = D / (WR * 16);
  static constexpr int RFA = RF2 > RF1 ? RF2 : RF1;
  // unpadded rows, swizzled (swz_off): D / 8 and FC / 8 units
  static constexpr int YSTR = D * 2, GSTR = FC * 2;
  static constexpr int YM = (D / 8 >= 16 ? 16 : D / 8) - 1, GM = (FC / 8 >= 16 ? 16 : FC / 8) - 1;
  static constexpr int KD = D / 32, KC = FC / 32;
  static constexpr int NB2 = D / 16;
  static constexpr int NGV = RF1 * NFC * 4;  // GELU values per lane per chunk
  static constexpr int LDS = MB * YSTR + 2 * MB * GSTR + MB * (2 * 4 * 4 + 8);
  // weight fragments (L2) requested PDA steps ahead, activation fragments
  // (LDS) PDB steps ahead: one each for wide window tiles; the 32-window
  // tiles of the update path have only two MFMAs per GEMM1 step and need more
  static constexpr bool SHORT = MB / WC_ <= 32;
  static constexpr int PDA = SHORT ? 4 : 1, PDB = SHORT ? 2 : 1;
};

struct PipeLane {
  __amdgpu_buffer_rsrc_t W1r, W2r;  // buffer descriptors of the packed W1 / W2 copies
  int w1o, w2o;                     // byte offset of this wave's first fragment column (wave-uniform)
  int NB1, lg, f0;
  int voff;                         // lane * 16 bytes
  const unsigned char* ybase;       // Ys row (m0 + lc)
  int yo[4], go[4];                 // swizzled fragment offsets in Ys / Gs rows (swz_off)
  int gwo[2];                       // swizzled offset of this lane's GELU values rf = 0, 1 in a Gs row
};

// Buffer descriptor over n bytes at p (raw, untyped; reads past n return 0).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* p, int64_t n) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)n, 0x00020000);
}
// The lane's 16-byte fragment at a wave-uniform byte offset: one buffer load
// with the lane offset in a vector register and the rest in a scalar one.
__device__ __forceinline__ uint4 frag_at(__amdgpu_buffer_rsrc_t r, int voff, int soff) {
  return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0));
}

// Calls f(integral_constant<I>) for I = B .. E-1: every index is a constant.
template <int B, int E, class Fn>
__device__ __forceinline__ void static_for(Fn&& f) {
  if constexpr (B < E) {
    f(std::integral_constant<int, B>{});
    static_for<B + 1, E>(f);
  }
}

// One interval.  G2ON: GEMM2 of the chunk at feature c2 from buffer gr;
// G1ON: GEMM1 of the chunk at feature c1 into un; GELUON: GELU of ug into gw.
template <int D, int MB, int WC, bool G2ON, bool G1ON, bool GELUON>
__device__ __forceinline__ void ffn_interval(const PipeLane& L,
                                             f32x4 (&y)[FfnPipe<D, MB, WC>::RF2][FfnPipe<D, MB, WC>::NFC],
                                             f32x4 (&ug)[FfnPipe<D, MB, WC>::RF1][FfnPipe<D, MB, WC>::NFC],
                                             f32x4 (&un)[FfnPipe<D, MB, WC>::RF1][FfnPipe<D, MB, WC>::NFC], int c1, int c2,
                                             const unsigned char* gr, unsigned char* gw) {
  typedef FfnPipe<D, MB, WC> P;
  constexpr int NFC = P::NFC, RF1 = P::RF1, RF2 = P::RF2, RFA = P::RFA;
  constexpr int S2 = G2ON ? P::KC : 0, S1 = G1ON ? P::KD : 0, NS = S2 + S1;
  constexpr int NM = S2 * RF2 * NFC + S1 * RF1 * NFC;
  constexpr int NGV = GELUON ? P::NGV : 0;
  static_assert(NS > 0, "empty interval");
  if constexpr (G1ON) {
#pragma unroll
    for (int rf = 0; rf < RF1; ++rf)
#pragma unroll
      for (int nf = 0; nf < NFC; ++nf) un[rf][nf] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  const int kc2 = c2 / 32, nb1 = c1 / 16;
  constexpr int PDA = P::PDA, NA = PDA + 1, PDB = P::PDB, NB = PDB + 1;
  uint4 A[NA][RFA], B[NB][NFC];
  auto loadA = [&](auto sc) {
    constexpr int s = decltype(sc)::value, buf = s % NA;
    if constexpr (s < S2) {
#pragma unroll
      for (int rf = 0; rf < RF2; ++rf) A[buf][rf] = frag_at(L.W2r, L.voff, L.w2o + ((kc2 + s) * P::NB2 + rf) * 1024);
    } else {
      constexpr int ks = s - S2;
#pragma unroll
      for (int rf = 0; rf < RF1; ++rf) A[buf][rf] = frag_at(L.W1r, L.voff, L.w1o + (ks * L.NB1 + nb1 + rf) * 1024);
    }
  };
  auto loadB = [&](auto sc) {
    constexpr int s = decltype(sc)::value, buf = s % NB;
    if constexpr (s < S2) {
#pragma unroll
      for (int nf = 0; nf < NFC; ++nf) B[buf][nf] = *(const uint4*)(gr + nf * 16 * P::GSTR + L.go[s & 3]);
    } else {
      constexpr int ks = s - S2;
#pragma unroll
      for (int nf = 0; nf < NFC; ++nf)
        B[buf][nf] = *(const uint4*)(L.ybase + nf * 16 * P::YSTR + (ks & ~3) * 64 + L.yo[ks & 3]);
    }
  };
  static_for<0, (PDA < NS ? PDA : NS)>(loadA);
  static_for<0, (PDB < NS ? PDB : NS)>(loadB);
  static_for<0, NS>([&](auto sc) {
    constexpr int s = decltype(sc)::value, abuf = s % NA, bbuf = s % NB;
    if constexpr (s + PDA < NS) loadA(std::integral_constant<int, s + PDA>{});
    if constexpr (s + PDB < NS) loadB(std::integral_constant<int, s + PDB>{});
    constexpr bool g2 = s < S2;
    constexpr int RFN = g2 ? RF2 : RF1;
    constexpr int MB0 = g2 ? s * RF2 * NFC : S2 * RF2 * NFC + (s - S2) * RF1 * NFC;
    static_for<0, RFN * NFC>([&](auto ic) {
      constexpr int i = decltype(ic)::value, rf = i / NFC, nf = i % NFC, m = MB0 + i;
      if constexpr (g2)
        Mma<true>::run(y[rf][nf], A[abuf][rf], B[bbuf][nf]);
      else
        Mma<true>::run(un[rf][nf], A[abuf][rf], B[bbuf][nf]);
      if constexpr (NGV > 0) {
        static_for<(m * NGV) / NM, ((m + 1) * NGV) / NM>([&](auto gc) {
          constexpr int g = decltype(gc)::value;
          f32x4& v = ug[g / (NFC * 4)][(g / 4) % NFC];
          v[g % 4] = gelu2_ex(v[g % 4]);
        });
      }
    });
    // the step's loads first, then each MFMA followed by a share of the vector work
    __builtin_amdgcn_sched_group_barrier(0x020, RFA, 0);
    __builtin_amdgcn_sched_group_barrier(0x100, NFC, 0);
    static_for<0, RFN * NFC>([&](auto) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x002, 3, 0);
    });
    // keep each step's loads one step ahead, not hoisted further
    __builtin_amdgcn_sched_barrier(0);
  });
  if constexpr (GELUON) {
#pragma unroll
    for (int nf = 0; nf < NFC; ++nf)
#pragma unroll
      for (int rf = 0; rf < RF1; ++rf)
        put4((uint16_t*)(gw + nf * 16 * P::GSTR + L.gwo[rf]), ug[rf][nf]);
  }
}

template <int D, int MB, bool KEEP, int WC>
__global__ __launch_bounds__(512) void k_ffn_pipe(FfnArgs a) {
  typedef FfnPipe<D, MB, WC> P;
  constexpr int NFC = P::NFC, RF1 = P::RF1, RF2 = P::RF2, FC = P::FC;
  static_assert(RF1 >= 1 && RF2 >= 1 && NFC >= 1 && MB % (16 * P::WC) == 0, "shape");
  static_assert(P::LDS <= 160 * 1024, "LDS");
  __shared__ __align__(16) unsigned char Ys[MB * P::YSTR];
  __shared__ __align__(16) unsigned char Gs[2][MB * P::GSTR];
  __shared__ float red[2][4][MB];
  __shared__ float zy[MB];
  __shared__ int tg[MB];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, lg = lane >> 4, lc = lane & 15;
  const int wr = wave % P::WR, wc = wave / P::WR;
  const int64_t tile0 = (int64_t)blockIdx.x * MB;
  const int64_t N = a.w.N;
  const int F = a.F;
  const int NC = F / FC;  // even: F is a multiple of 256
  const int m0 = wc * P::CW;
  const int d0 = wr * (D / P::WR);
  PipeLane L;
  L.f0 = __builtin_amdgcn_readfirstlane(wr * (FC / P::WR));
  L.W1r = make_rsrc(a.W1, (int64_t)D * F * 2 * (a.wstride ? a.k : 1));
  L.W2r = make_rsrc(a.W2, (int64_t)D * F * 2 * (a.wstride ? a.k : 1));
  L.w1o = (L.f0 / 16) * 1024;
  L.w2o = __builtin_amdgcn_readfirstlane(d0 / 16) * 1024;
  L.NB1 = F / 16;
  L.voff = lane * 16;
  L.lg = lg;
  L.ybase = Ys + (m0 + lc) * P::YSTR;
  swz_off(lg, lc, P::YM, L.yo);
  swz_off(lg, lc, P::GM, L.go);
#pragma unroll
  for (int rf = 0; rf < 2; ++rf) L.gwo[rf] = swz_elem(lc, L.f0 + rf * 16 + 4 * lg, P::GM);
  const unsigned char* gr0 = Gs[0] + (m0 + lc) * P::GSTR;
  const unsigned char* gr1 = Gs[1] + (m0 + lc) * P::GSTR;
  unsigned char* gw0 = Gs[0] + (m0 + lc) * P::GSTR;
  unsigned char* gw1 = Gs[1] + (m0 + lc) * P::GSTR;

  f32x4 y[RF2][NFC];
#pragma unroll
  for (int nf = 0; nf < NFC; ++nf) {
    const int64_t n = tile0 + m0 + nf * 16 + lc;
#pragma unroll
    for (int rf = 0; rf < RF2; ++rf) {
      if (n < N) {
        const float4 v = *reinterpret_cast<const float4*>(a.h0 + n * D + d0 + rf * 16 + 4 * lg);
        y[rf][nf] = f32x4{v.x, v.y, v.z, v.w};
      } else {
        y[rf][nf] = f32x4{0.f, 0.f, 0.f, 0.f};
      }
    }
  }
  if (tid < MB) {
    const int64_t n = tile0 + tid;
    int v = 0;
    if (n < N) {
      v = a.w.streams[target_offset(a.w, n)];
      if (KEEP) a.ktgt[n] = v;
    }
    tg[tid] = v;
  }

  f32x4 ua[RF1][NFC], ub[RF1][NFC];
  // pre-GELU U of the chunk at feature c, kept for the backward pass
  auto keep_u = [&](const f32x4 (&u)[RF1][NFC], int rep, int c) {
#pragma unroll
    for (int nf = 0; nf < NFC; ++nf) {
      const int64_t n = tile0 + m0 + nf * 16 + lc;
      if (n < N) {
#pragma unroll
        for (int rf = 0; rf < RF1; ++rf)
          *reinterpret_cast<float4*>(a.kU + ((int64_t)rep * N + n) * F + c + L.f0 + rf * 16 + 4 * lg) =
              make_float4(u[rf][nf][0], u[rf][nf][1], u[rf][nf][2], u[rf][nf][3]);
      }
    }
  };

  // GELU of the chunk at feature c (held doubled after its interval), kept as
  // the bf16 operand values the second product used
  auto keep_g = [&](const f32x4 (&g)[RF1][NFC], int rep, int c) {
#pragma unroll
    for (int nf = 0; nf < NFC; ++nf) {
      const int64_t n = tile0 + m0 + nf * 16 + lc;
      if (n < N) {
#pragma unroll
        for (int rf = 0; rf < RF1; ++rf)
          *reinterpret_cast<uint2*>(a.kG + ((int64_t)rep * N + n) * F + c + L.f0 + rf * 16 + 4 * lg) =
              make_uint2(pack_bf16x2(0.5f * round_bf(g[rf][nf][0]), 0.5f * round_bf(g[rf][nf][1])),
                         pack_bf16x2(0.5f * round_bf(g[rf][nf][2]), 0.5f * round_bf(g[rf][nf][3])));
      }
    }
  };

  const int w1o0 = L.w1o, w2o0 = L.w2o;  // repeat 0's fragment offsets
  for (int rep = 0; rep <= a.k; ++rep) {
    // untied FFN: repeat rep's copies (wstride uint4 further per repeat)
    L.w1o = w1o0 + (rep < a.k ? rep : 0) * (int)(a.wstride * 16);
    L.w2o = w2o0 + (rep < a.k ? rep : 0) * (int)(a.wstride * 16);
#pragma unroll
    for (int nf = 0; nf < NFC; ++nf) {
      const int m = m0 + nf * 16 + lc;
      const int64_t n = tile0 + m;
#pragma unroll
      for (int rf = 0; rf < RF2; ++rf) {
        const int dd = d0 + rf * 16 + 4 * lg;
        if (KEEP && n < N) put4((uint16_t*)a.kY + ((int64_t)rep * N + n) * D + dd, y[rf][nf]);
        put4((uint16_t*)(Ys + m * P::YSTR + swz_elem(m, dd, P::YM)), y[rf][nf]);
      }
    }
    __syncthreads();
    if (rep == a.k) break;
    // prologue: GEMM1 of chunk 0 into ua
    ffn_interval<D, MB, WC, false, true, false>(L, y, ub, ua, 0, 0, gr0, gw0);
    if (KEEP) keep_u(ua, rep, 0);
    // j = 0: GELU(0) -> buffer 0, GEMM1(1) -> ub
    ffn_interval<D, MB, WC, false, true, true>(L, y, ua, ub, FC, 0, gr0, gw0);
    if (KEEP) keep_g(ua, rep, 0);
    __syncthreads();
    for (int j = 1; j < NC - 1; j += 2) {
      if (KEEP) keep_u(ub, rep, j * FC);
      // j (odd): GELU(j) -> buffer 1, GEMM1(j+1) -> ua, GEMM2(j-1) from buffer 0
      ffn_interval<D, MB, WC, true, true, true>(L, y, ub, ua, (j + 1) * FC, (j - 1) * FC, gr0, gw1);
      if (KEEP) keep_g(ub, rep, j * FC);
      __syncthreads();
      if (KEEP) keep_u(ua, rep, (j + 1) * FC);
      // j+1 (even): GELU(j+1) -> buffer 0, GEMM1(j+2) -> ub, GEMM2(j) from buffer 1
      ffn_interval<D, MB, WC, true, true, true>(L, y, ua, ub, (j + 2) * FC, j * FC, gr1, gw0);
      if (KEEP) keep_g(ua, rep, (j + 1) * FC);
      __syncthreads();
    }
    if (KEEP) keep_u(ub, rep, (NC - 1) * FC);
    // j = NC-1 (odd): GELU(NC-1) -> buffer 1, GEMM2(NC-2) from buffer 0
    ffn_interval<D, MB, WC, true, false, true>(L, y, ub, ua, 0, (NC - 2) * FC, gr0, gw1);
    if (KEEP) keep_g(ub, rep, (NC - 1) * FC);
    __syncthreads();
    // epilogue: GEMM2(NC-1) from buffer 1
    ffn_interval<D, MB, WC, true, false, false>(L, y, ua, ub, 0, (NC - 1) * FC, gr1, gw0);
  }
  ffn_head_out<true, D, MB, KEEP, P::YSTR, P::YM>(a, Ys, red, zy, tg);
}

// ------------------------------------------------------------ dispatch ----
// bf16 runs the pipelined kernel (k_ffn_pipe); fp32 runs k_ffn_head.
// Measured on the main workload (2^20 windows, d = 256), k_ffn_head in bf16
// took 3.67 ms and k_ffn_pipe 3.55 ms.  Slower alternatives measured: two 4-wave
// workgroups of 64 windows per CU (each window carries twice the weight traffic
// from L2), 4.5 ms; the pipeline with weights requested 2 or 3 steps ahead
// instead of 1, 3.65 / 3.69 ms; LDS row padding of 32 or 64 bytes instead of 16,
// 3.60 / 3.84 ms (none: 6.25 ms); the same pipeline on v_mfma_f32_32x32x16_bf16
// tiles, 3.71-3.79 ms against 3.62-3.65 ms: it takes 8.5% fewer cycles, but the
// clock under load falls from 1.98 to 1.84 GHz.  This kernel runs at the power
// limit: a loop of MFMAs alone on random bf16 operands sustains 1.94-2.04 PF/s
// with 16x16x32 and 1.53 PF/s with 32x32x16 (2.41 / 2.44 PF/s on constant ones).
constexpr int ffn_lds_bytes(bool bf, int D, int mb, int fc) {
  return mb * (D * (bf ? 2 : 4) + 16) + mb * (fc * (bf ? 2 : 4) + 16) + mb * (2 * 4 * 4 + 8);
}
// largest window tile, then widest F chunk, that fits the 160 KiB of LDS
constexpr int pick_mb(bool bf, int D) {
  return ffn_lds_bytes(bf, D, 128, 128) <= 160 * 1024 ? 128 : ffn_lds_bytes(bf, D, 64, 128) <= 160 * 1024 ? 64 : 32;
}
constexpr int pick_fc(bool bf, int D) { return ffn_lds_bytes(bf, D, pick_mb(bf, D), 256) <= 160 * 1024 ? 256 : 128; }

template <int D>
constexpr int pick_mb_pipe() { return FfnPipe<D, 128>::LDS <= 160 * 1024 ? 128 : 64; }

template <int D, int MB, int WC = 2>
static void launch_pipe(const FfnArgs& a, hipStream_t s) {
  static_assert(FfnPipe<D, MB, WC>::LDS <= 160 * 1024, "LDS");
  const dim3 grid((unsigned)((a.w.N + MB - 1) / MB));
  if (a.kY)
    hipLaunchKernelGGL((k_ffn_pipe<D, MB, true, WC>), grid, dim3(512), 0, s, a);
  else
    hipLaunchKernelGGL((k_ffn_pipe<D, MB, false, WC>), grid, dim3(512), 0, s, a);
}

template <bool BF, int D>
static void run_ffn(const FfnArgs& a, hipStream_t s) {
  if constexpr (BF) {
    // the widest window tile that still gives every CU a workgroup; launches of
    // a few thousand windows (one step of the update path) take 32-window tiles
    constexpr int MB = pick_mb_pipe<D>();
    // tiles of up to 64 windows put all 8 waves across the features (each
    // weight fragment read once per block; measured 14% faster at d = 512);
    // 128-window tiles split the waves 4 x 2 (fewer LDS reads per MFMA)
    constexpr int WCB = (MB <= 64 && D >= 128) ? 1 : 2;
    if (a.w.N >= (int64_t)256 * MB)
      launch_pipe<D, MB, WCB>(a, s);
    else if constexpr (D >= 128)
      launch_pipe<D, 32, 1>(a, s);
    else
      launch_pipe<D, 32>(a, s);
  } else {
    constexpr int MB = pick_mb(BF, D), FC = pick_fc(BF, D);
    static_assert(ffn_lds_bytes(BF, D, MB, FC) <= 160 * 1024, "LDS");
    const dim3 grid((unsigned)((a.w.N + MB - 1) / MB));
    if (a.kY)
      hipLaunchKernelGGL((k_ffn_head<BF, D, MB, FC, true>), grid, dim3(512), 0, s, a);
    else
      hipLaunchKernelGGL((k_ffn_head<BF, D, MB, FC, false>), grid, dim3(512), 0, s, a);
  }
}

ffn_fn find_ffn(bool bf, int D) {
#define TRACE_FFN(BF_, D_) \
  if (bf == BF_ && D == D_) return &run_ffn<BF_, D_>;
  TRACE_FFN(true, 64) TRACE_FFN(true, 128) TRACE_FFN(true, 256) TRACE_FFN(true, 512)
  TRACE_FFN(false, 64) TRACE_FFN(false, 128) TRACE_FFN(false, 256) TRACE_FFN(false, 512)
#undef TRACE_FFN
  return nullptr;
}
