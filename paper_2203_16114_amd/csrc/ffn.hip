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
// MFMAs that use them; the activations are read from LDS.
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
  const uint4* __restrict__ W1p = a.W1;
  const uint4* __restrict__ W2p = a.W2;

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
#pragma unroll
    for (int nf = 0; nf < NFC; ++nf) {
      const int m = m0 + nf * 16 + lc;
      const int64_t n = tile0 + m;
#pragma unroll
      for (int rf = 0; rf < RF2; ++rf) {
        const int dd = d0 + rf * 16 + 4 * lg;
        if (KEEP && n < N)
          *reinterpret_cast<float4*>(a.kY + ((int64_t)rep * N + n) * D + dd) =
              make_float4(y[rf][nf][0], y[rf][nf][1], y[rf][nf][2], y[rf][nf][3]);
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
          for (int rf = 0; rf < RF1; ++rf) wa[0][rf] = W1p[(nb1n + rf) * 64 + lane];
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

  // head on bf(Y_k) (staged in Ys by the last pass above)
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
    for (int nf = 0; nf < NFC; ++nf) bb[nf] = *(const uint4*)(yrow[nf] + ks * 64);
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
    float se = 0.f;
#pragma unroll
    for (int rf = 0; rf < RFH; ++rf)
#pragma unroll
      for (int r = 0; r < 4; ++r) se += expf(z[rf][nf][r] - mx);
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

// ------------------------------------------------------------ dispatch ----
// Measured alternatives, both slower on the main workload (2^20 windows):
// two 4-wave workgroups of 64 windows per CU (barriers desynchronised, but each
// window carries twice the weight traffic from L2): 4.5 ms against 3.8 ms; a
// software pipeline with G double-buffered in LDS (GEMM2 of chunk c, GELU of
// chunk c+1 and GEMM1 of chunk c+2 in one interval), which needs 128-feature
// chunks to fit the LDS: 4.5 ms.
constexpr int ffn_lds_bytes(bool bf, int D, int mb, int fc) {
  return mb * (D * (bf ? 2 : 4) + 16) + mb * (fc * (bf ? 2 : 4) + 16) + mb * (2 * 4 * 4 + 8);
}
// largest window tile, then widest F chunk, that fits the 160 KiB of LDS
constexpr int pick_mb(bool bf, int D) {
  return ffn_lds_bytes(bf, D, 128, 128) <= 160 * 1024 ? 128 : ffn_lds_bytes(bf, D, 64, 128) <= 160 * 1024 ? 64 : 32;
}
constexpr int pick_fc(bool bf, int D) { return ffn_lds_bytes(bf, D, pick_mb(bf, D), 256) <= 160 * 1024 ? 256 : 128; }

template <bool BF, int D>
static void run_ffn(const FfnArgs& a, hipStream_t s) {
  constexpr int MB = pick_mb(BF, D), FC = pick_fc(BF, D);
  static_assert(ffn_lds_bytes(BF, D, MB, FC) <= 160 * 1024, "LDS");
  const dim3 grid((unsigned)((a.w.N + MB - 1) / MB));
  if (a.kY)
    hipLaunchKernelGGL((k_ffn_head<BF, D, MB, FC, true>), grid, dim3(512), 0, s, a);
  else
    hipLaunchKernelGGL((k_ffn_head<BF, D, MB, FC, false>), grid, dim3(512), 0, s, a);
}

ffn_fn find_ffn(bool bf, int D) {
#define TRACE_FFN(BF_, D_) \
  if (bf == BF_ && D == D_) return &run_ffn<BF_, D_>;
  TRACE_FFN(true, 64) TRACE_FFN(true, 128) TRACE_FFN(true, 256) TRACE_FFN(true, 512)
  TRACE_FFN(false, 64) TRACE_FFN(false, 128) TRACE_FFN(false, 256) TRACE_FFN(false, 512)
#undef TRACE_FFN
  return nullptr;
}
