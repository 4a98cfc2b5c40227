// Byte-grouping gather (Sec. 4.2) and the causal multi-head attention of the
// last token (Eqs. 1-2) with its output projection and the first residual of
// Eq. 4, fused: window bytes -> h0 = O.Wo + X_last.
//
// One workgroup of 8 waves per tile of MA windows.  Wave w owns RFW*16
// consecutive token rows (whole windows).  The byte-embedding part of its
// tokens stays in registers for the whole kernel as MFMA B-operand fragments
// (8 consecutive features per lane); the positional part enters every
// projection as a precomputed row of P.W (X.W = E.W + P.W, X = E + P in fp32).
// Every product is formed transposed (weights as the A operand), so a lane's
// four results are four consecutive features of one token:
//   q^T   = Wq^T . E_last^T + (P.Wq)[T-1]   (waves split the features)   -> LDS
//   per head h:  K_h^T = Wk_h^T . X^T, then V_h^T = Wv_h^T . X^T; the head's
//                weight fragments are staged through LDS in double-buffered
//                chunks shared by all 8 waves, moved by direct global-to-LDS
//                loads issued one chunk ahead;
//                score of row u = q . K_u / sqrt(dh): 4-lane-group reduction;
//                softmax over the T rows of a window and O_h = sum_u a_u V_u:
//                DPP reductions over the T lanes that hold one window  -> LDS
//   h0^T  = Wo^T . O^T + X_last (fp32)    (waves split the features)   -> HBM
// Only the last query row is formed: the head reads the last token, and under
// the causal mask that row attends to every key of the window.
#include "kcommon.h"
#include "kernels.h"
#include "win.h"

namespace {

// E-part of a token fragment: features [d, d + EPF) of token t of a window
// whose bytes are at wb, one 16-byte load from the byte embedding (the
// positional part enters the projections through the table P.W).
template <bool BF>
__device__ __forceinline__ uint4 x_frag(const typename Mma<BF>::T* __restrict__ E, const uint8_t* wb, int t, int d,
                                        int e, int g, uint32_t einv) {
  const int j = (int)(((uint32_t)d * einv) >> 20), cc = d - j * e;
  const int byte = wb[t * g + j];
  return *reinterpret_cast<const uint4*>(E + byte * e + cc);
}

// A token fragment from an input row of a later layer: EPF consecutive fp32
// values at X + i (i < 0: a dead window, zeros), as the operand type.
template <bool BF>
__device__ __forceinline__ uint4 x_row_frag(const float* __restrict__ X, int64_t i) {
  if (i < 0) return make_uint4(0u, 0u, 0u, 0u);
  const float4 lo = *reinterpret_cast<const float4*>(X + i);
  if constexpr (BF) {
    const float4 hi = *reinterpret_cast<const float4*>(X + i + 4);
    return make_uint4(pack_bf16x2(lo.x, lo.y), pack_bf16x2(lo.z, lo.w), pack_bf16x2(hi.x, hi.y),
                      pack_bf16x2(hi.z, hi.w));
  } else {
    return make_uint4(__float_as_uint(lo.x), __float_as_uint(lo.y), __float_as_uint(lo.z), __float_as_uint(lo.w));
  }
}

__device__ __forceinline__ void put4o(uint16_t* p, const f32x4& v) {
  *reinterpret_cast<uint2*>(p) = make_uint2(pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]));
}
__device__ __forceinline__ void put4o(float* p, const f32x4& v) {
  *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
}
__device__ __forceinline__ f32x4 rounded4(const f32x4& v, bool bf) {
  if (!bf) return v;
  return f32x4{round_bf(v[0]), round_bf(v[1]), round_bf(v[2]), round_bf(v[3])};
}

// Performer (FAVOR+) weight of key row u of a window's last query, for one
// head: phi(q')^T phi(k'_u) normalised over the window's T rows, with
// phi(x) = exp(omega x - |x|^2/2), q' = q dh^-1/4, k' = k dh^-1/4 (the
// 1/sqrt(m) factor cancels).  phi(q')^T phi(k'_u) = sum_i exp(omega_i w -
// (|q'|^2 + |k'_u|^2)/2) with w = q' + k'_u.  The lane holds row u's key as an
// accumulator quad per 16 columns (c = 16 f + 4 lg + r) and reads q from its
// LDS row; w becomes the B operand of the projection in that same order (one
// fp32 fragment per quad, or in bf16 a hi and a lo fragment per two quads,
// matched by the packing of omega), so each 16-feature block is one MFMA chain
// whose result gives the lane features 4 lg + r of row u.  The sum over
// features runs with a running maximum (base 2); the maximum over the window
// is subtracted before the rows are normalised (it cancels).
template <bool BF, int T, int NFH>
__device__ __forceinline__ float perf_weight(const f32x4 (&k)[NFH], const float* __restrict__ qrow, int lg,
                                             const uint4* __restrict__ Om, int nfeat, float s4) {
  typedef Mma<BF> M;
  constexpr int KST = BF ? NFH / 2 : NFH;  // k-steps over the head width
  float w[NFH][4];
  float nrm = 0.f;
#pragma unroll
  for (int f = 0; f < NFH; ++f) {
    const float4 q4 = *reinterpret_cast<const float4*>(qrow + f * 16 + 4 * lg);
    const float qv[4] = {q4.x, q4.y, q4.z, q4.w};
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      nrm = fmaf(k[f][r], k[f][r], fmaf(qv[r], qv[r], nrm));
      w[f][r] = s4 * (qv[r] + k[f][r]);
    }
  }
  nrm += __shfl_xor(nrm, 16, 64);
  nrm += __shfl_xor(nrm, 32, 64);
  const float base = -0.5f * s4 * s4 * nrm * TRACE_LOG2E;  // -(|q'|^2 + |k'|^2)/2, base 2
  uint4 bh[KST], bl[KST];
#pragma unroll
  for (int st = 0; st < KST; ++st) {
    if constexpr (BF) {
      float hv[8], lv[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const float x = j < 4 ? w[2 * st][j] : w[2 * st + 1][j - 4];
        hv[j] = round_bf(x);
        lv[j] = x - hv[j];
      }
      bh[st] = make_uint4(pack_bf16x2(hv[0], hv[1]), pack_bf16x2(hv[2], hv[3]), pack_bf16x2(hv[4], hv[5]),
                          pack_bf16x2(hv[6], hv[7]));
      bl[st] = make_uint4(pack_bf16x2(lv[0], lv[1]), pack_bf16x2(lv[2], lv[3]), pack_bf16x2(lv[4], lv[5]),
                          pack_bf16x2(lv[6], lv[7]));
    } else {
      bh[st] = make_uint4(__float_as_uint(w[st][0]), __float_as_uint(w[st][1]), __float_as_uint(w[st][2]),
                          __float_as_uint(w[st][3]));
      bl[st] = bh[st];
    }
  }
  const int lane = threadIdx.x & 63;
  float mx = 0.f, sm = 0.f;
  for (int b = 0; b < nfeat / 16; ++b) {
    f32x4 z = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int st = 0; st < KST; ++st) {
      const uint4 om = Om[(b * KST + st) * 64 + lane];
      M::run(z, om, bh[st]);
      if constexpr (BF) M::run(z, om, bl[st]);
    }
    float x[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) x[r] = fmaf(z[r], TRACE_LOG2E, base);
    const float bm = fmaxf(fmaxf(x[0], x[1]), fmaxf(x[2], x[3]));
    const float nm = b == 0 ? bm : fmaxf(mx, bm);
    float acc = b == 0 ? 0.f : sm * __builtin_amdgcn_exp2f(mx - nm);
#pragma unroll
    for (int r = 0; r < 4; ++r) acc += __builtin_amdgcn_exp2f(x[r] - nm);
    sm = acc;
    mx = nm;
  }
  // the row's four lane groups hold different features: combine them
#pragma unroll
  for (int off = 16; off <= 32; off <<= 1) {
    const float om = __shfl_xor(mx, off, 64), os = __shfl_xor(sm, off, 64);
    const float nm = fmaxf(mx, om);
    sm = sm * __builtin_amdgcn_exp2f(mx - nm) + os * __builtin_amdgcn_exp2f(om - nm);
    mx = nm;
  }
  const float wmax = group_max<T>(mx);
  const float sc = sm * __builtin_amdgcn_exp2f(mx - wmax);
  return sc * __builtin_amdgcn_rcpf(group_sum<T>(sc));
}

template <bool BF, int T, int D, int DH, bool SMALL = false>
struct AttnShape {
  typedef typename Mma<BF>::T OT;
  static constexpr int NW = 8;
  static constexpr int KSTEPS = D / Mma<BF>::KS;
  static constexpr int NFH = DH / 16;
  static constexpr int KSC = (KSTEPS * NFH <= 16) ? KSTEPS : 16 / NFH;  // k-steps per staged chunk
  static constexpr int CHUNK = KSC * NFH * 64;                            // uint4 per chunk
  static constexpr int XLSTR = D * (int)sizeof(OT) + 16;
  static constexpr int lds(int rfw) {
    return 2 * CHUNK * 16 + (NW * rfw * 16 / T) * (D * 4 + XLSTR + 64) + 2 * 2 * T * DH * 4;
  }
  // row fragments per wave: the largest of 4, 2, 1 whose register-held tokens,
  // accumulators and fragments stay within the register budget of two waves per
  // SIMD and whose tile fits the LDS
  static constexpr int vgprs(int rfw) { return rfw * KSTEPS * 4 + rfw * NFH * 4 + NFH * 4 + 8; }
  static constexpr bool fits(int rfw) { return vgprs(rfw) <= 184 && lds(rfw) <= 160 * 1024; }
  static constexpr int RFW = SMALL ? 1 : (KSTEPS <= 8 && fits(4)) ? 4 : (fits(2) ? 2 : 1);
  static constexpr int RW = RFW * 16;
  static constexpr int MA = NW * RW / T;
  static constexpr int LDS = lds(RFW);
};

}  // namespace

template <bool BF, int T, int D, int DH, bool KEEP, bool SMALL, bool PERF>
__global__ __launch_bounds__(512) void k_attn(AttnArgs a) {
  typedef Mma<BF> M;
  typedef typename M::T OT;
  typedef AttnShape<BF, T, D, DH, SMALL> S;
  constexpr int H = D / DH;
  constexpr int NW = S::NW, KSTEPS = S::KSTEPS, NFH = S::NFH, KSC = S::KSC, CPP = KSTEPS / KSC, CHUNK = S::CHUNK;
  constexpr int RFW = S::RFW, RW = S::RW, MA = S::MA, XLSTR = S::XLSTR;
  constexpr int NQF = D / 16, QFW = (NQF + NW - 1) / NW, NMF = (MA + 15) / 16;
  constexpr int NB = D / 16;
  static_assert(KSTEPS % KSC == 0 && (T == 4 || T == 8) && MA % 16 == 0, "shape");
  __shared__ uint4 Wst[2][CHUNK];
  __shared__ __align__(16) float Qs[MA * D];
  __shared__ __align__(16) unsigned char Xl[MA * XLSTR];  // X_last rows, then O rows
  __shared__ uint8_t Wb[MA * 64];
  __shared__ __align__(16) float PKV[2][2][T * DH];  // head slices of P.Wk and P.Wv, double-buffered

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, lg = lane >> 4, lc = lane & 15;
  const int64_t tile0 = (int64_t)blockIdx.x * MA;
  const int64_t N = a.w.N;
  const int W = T * a.g;
  const OT* __restrict__ E = (const OT*)a.E;
  const OT* __restrict__ P = (const OT*)a.P;
  const float* __restrict__ PQ = a.PW;  // [T][D] each: P.Wq, P.Wk, P.Wv
  const float* __restrict__ PK = a.PW + (int64_t)T * D;
  const float* __restrict__ PV = a.PW + (int64_t)2 * T * D;

  // window bytes to LDS: wave w takes windows w, w + 8, ... (one offset per
  // window, on the scalar unit), lane j < W takes byte j
  for (int m = __builtin_amdgcn_readfirstlane(wave); m < MA; m += NW) {
    const int64_t n = tile0 + m;
    if (lane < W) {
      uint8_t v = 0;
      if (n < N) {
        v = a.w.streams[target_offset(a.w, n) - W + lane];
        if (KEEP) a.kwin[n * W + lane] = v;
      }
      Wb[m * 64 + lane] = v;
    }
  }
  // d / e as (d * einv) >> 20: exact for d < 1024 and e < 2048
  const uint32_t einv = ((1u << 20) + (uint32_t)a.e - 1u) / (uint32_t)a.e;
  __syncthreads();

  // this wave's tokens as B fragments; the last token of each window also to LDS
  uint4 xb[RFW][KSTEPS];
#pragma unroll
  for (int rf = 0; rf < RFW; ++rf) {
    const int row = wave * RW + rf * 16 + lc;
    const int m = row / T, t = row - m * T;
#pragma unroll
    for (int ks = 0; ks < KSTEPS; ++ks) {
      const int d = ks * M::KS + lg * M::EPF;
      if (a.Xin)  // a later layer: its input rows, as operands (bf16: rounded)
        xb[rf][ks] = x_row_frag<BF>(a.Xin, tile0 + m < N ? ((tile0 + m) * T + t) * D + d : -1);
      else
        xb[rf][ks] = x_frag<BF>(E, Wb + m * 64, t, d, a.e, a.g, einv);
      if (t == T - 1) *(uint4*)(Xl + m * XLSTR + ks * 64 + lg * 16) = xb[rf][ks];
    }
  }
  __syncthreads();

  // q^T = Wq^T . X_last^T ; lane holds q[m = nf*16 + lc][c = qf*16 + 4*lg + r]
#pragma unroll
  for (int qi = 0; qi < QFW; ++qi) {
    const int qf = wave * QFW + qi;
    if (qf < NQF) {
      f32x4 acc[NMF];
#pragma unroll
      for (int nf = 0; nf < NMF; ++nf) acc[nf] = f32x4{0.f, 0.f, 0.f, 0.f};
      uint4 wq[2];
      wq[0] = a.Wq[qf * 64 + lane];
#pragma unroll
      for (int ks = 0; ks < KSTEPS; ++ks) {
        if (ks + 1 < KSTEPS) wq[(ks + 1) & 1] = a.Wq[((ks + 1) * NB + qf) * 64 + lane];
#pragma unroll
        for (int nf = 0; nf < NMF; ++nf) {
          const uint4 bx = *(const uint4*)(Xl + (nf * 16 + lc) * XLSTR + ks * 64 + lg * 16);
          M::run(acc[nf], wq[ks & 1], bx);
        }
      }
      const float4 pq = *reinterpret_cast<const float4*>(PQ + (T - 1) * D + qf * 16 + 4 * lg);
#pragma unroll
      for (int nf = 0; nf < NMF; ++nf) {
        const int m = nf * 16 + lc;
        const int c = qf * 16 + 4 * lg;
        acc[nf][0] += pq.x;
        acc[nf][1] += pq.y;
        acc[nf][2] += pq.z;
        acc[nf][3] += pq.w;
        *reinterpret_cast<float4*>(Qs + m * D + c) = make_float4(acc[nf][0], acc[nf][1], acc[nf][2], acc[nf][3]);
        if (KEEP && tile0 + m < N)
          *reinterpret_cast<float4*>(a.kq + (tile0 + m) * D + c) =
              make_float4(acc[nf][0], acc[nf][1], acc[nf][2], acc[nf][3]);
      }
    }
  }

  // staged weight chunks: chunk c = ((h * 2 + pass) * CPP + ck); element i of a
  // chunk is fragment (k-step ck*KSC + i/(NFH*64), feature frag h*NFH + (i/64)%NFH)
  auto chunk_src = [&](int c, int i) -> const uint4* {
    const int ck = c % CPP, pass = (c / CPP) & 1, h = c / (2 * CPP);
    const int kk = i / (NFH * 64), f = (i / 64) % NFH, ln = i & 63;
    const uint4* Wp = pass ? a.Wv : a.Wk;
    return Wp + ((ck * KSC + kk) * NB + h * NFH + f) * 64 + ln;
  };
  constexpr int NFRAG = KSC * NFH;  // fragments per chunk, 1 KiB each
  // chunk c -> LDS buffer: wave w moves fragments w, w + 8, ... with direct
  // global-to-LDS loads (16 bytes per lane, lane order), no register staging
  auto stage = [&](int c, int buf) {
#pragma unroll
    for (int q = wave; q < NFRAG; q += NW)
      __builtin_amdgcn_global_load_lds((const void*)chunk_src(c, q * 64 + lane),
                                       (__attribute__((address_space(3))) void*)(Wst[buf] + q * 64), 16, 0, 0);
  };
  constexpr int NCH = H * 2 * CPP;
  // rows t of P.Wk and P.Wv of head hh -> PKV[hh & 1] by direct 16-byte loads,
  // slot l = (which * T + t) * DH / 4 + c4
  constexpr int PKV_SLOTS = 2 * T * DH / 4;
  static_assert(PKV_SLOTS % 64 == 0, "PKV staging by whole waves");
  auto stage_pkv = [&](int hh) {
    if (wave * 64 < PKV_SLOTS) {
      const int l = wave * 64 + lane;
      const int which = l / (T * DH / 4), t = (l / (DH / 4)) % T, c4 = l % (DH / 4);
      const float* src = (which ? PV : PK) + t * D + hh * DH + 4 * c4;
      __builtin_amdgcn_global_load_lds((const void*)src,
                                       (__attribute__((address_space(3))) void*)(&PKV[hh & 1][0][0] + wave * 256), 16,
                                       0, 0);
    }
  };
  stage(0, 0);
  stage_pkv(0);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();  // chunk 0 and head 0's P rows staged; Qs complete; X_last rows no longer needed

  const float scale = a.scale;
  float prob[RFW];
  for (int h = 0; h < H; ++h) {
#pragma unroll
    for (int pass = 0; pass < 2; ++pass) {
      f32x4 acc[RFW][NFH];
#pragma unroll
      for (int rf = 0; rf < RFW; ++rf)
#pragma unroll
        for (int f = 0; f < NFH; ++f) acc[rf][f] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ck = 0; ck < CPP; ++ck) {
        const int c = (h * 2 + pass) * CPP + ck;
        if (c + 1 < NCH) stage(c + 1, (c + 1) & 1);
        const uint4* buf = Wst[c & 1];
#pragma unroll
        for (int kk = 0; kk < KSC; ++kk) {
          uint4 af[NFH];
#pragma unroll
          for (int f = 0; f < NFH; ++f) af[f] = buf[(kk * NFH + f) * 64 + lane];
#pragma unroll
          for (int rf = 0; rf < RFW; ++rf)
#pragma unroll
            for (int f = 0; f < NFH; ++f) M::run(acc[rf][f], af[f], xb[rf][ck * KSC + kk]);
        }
        __builtin_amdgcn_s_waitcnt(0);  // this wave's part of chunk c + 1 has landed
        __syncthreads();
        // every wave is past head h - 1, the last reader of PKV[(h + 1) & 1]:
        // stage head h + 1's P rows there (waited for at the next chunk barrier)
        if (pass == 0 && ck == 0 && h + 1 < H) stage_pkv(h + 1);
      }
      // lane holds K_h or V_h [row = wave*RW + rf*16 + lc][c = f*16 + 4*lg + r]
#pragma unroll
      for (int rf = 0; rf < RFW; ++rf) {
        const int row = wave * RW + rf * 16 + lc;
        const int m = row / T, t = row - m * T;
        const int64_t n = tile0 + m;
        const bool live = n < N;
        // positional part of the token's projection (this head's rows, staged in LDS)
        const float* pp = &PKV[h & 1][pass][0] + t * DH + 4 * lg;
#pragma unroll
        for (int f = 0; f < NFH; ++f) {
          const float4 p4 = *reinterpret_cast<const float4*>(pp + f * 16);
          acc[rf][f][0] += p4.x;
          acc[rf][f][1] += p4.y;
          acc[rf][f][2] += p4.z;
          acc[rf][f][3] += p4.w;
        }
        if (pass == 0) {
          if constexpr (PERF) {
            prob[rf] = perf_weight<BF, T, NFH>(acc[rf], Qs + m * D + h * DH, lg, a.Om, a.nfeat, a.scale4);
          } else {
            float s = 0.f;
#pragma unroll
            for (int f = 0; f < NFH; ++f) {
              const float4 q4 = *reinterpret_cast<const float4*>(Qs + m * D + h * DH + f * 16 + 4 * lg);
              s += q4.x * acc[rf][f][0] + q4.y * acc[rf][f][1] + q4.z * acc[rf][f][2] + q4.w * acc[rf][f][3];
            }
            s += __shfl_xor(s, 16, 64);
            s += __shfl_xor(s, 32, 64);
            s *= scale;
            const float mx = group_max<T>(s);
            const float p = expf(s - mx);
            const float sm = group_sum<T>(p);
            prob[rf] = p * __builtin_amdgcn_rcpf(sm);
          }
          if (KEEP && live) {
            if (lg == 0) a.kA[(n * H + h) * T + t] = prob[rf];
#pragma unroll
            for (int f = 0; f < NFH; ++f)
              *reinterpret_cast<float4*>(a.kK + (n * T + t) * D + h * DH + f * 16 + 4 * lg) =
                  make_float4(acc[rf][f][0], acc[rf][f][1], acc[rf][f][2], acc[rf][f][3]);
          }
        } else {
#pragma unroll
          for (int f = 0; f < NFH; ++f) {
            if (KEEP && live)
              *reinterpret_cast<float4*>(a.kV + (n * T + t) * D + h * DH + f * 16 + 4 * lg) =
                  make_float4(acc[rf][f][0], acc[rf][f][1], acc[rf][f][2], acc[rf][f][3]);
            f32x4 ov;
#pragma unroll
            for (int r = 0; r < 4; ++r) ov[r] = group_sum<T>(prob[rf] * acc[rf][f][r]);
            if (t == 0) {
              const int cc = h * DH + f * 16 + 4 * lg;
              put4o((OT*)(Xl + m * XLSTR) + cc, ov);
              if (KEEP && live) {
                const f32x4 rv = rounded4(ov, BF);
                *reinterpret_cast<float4*>(a.kO + n * D + cc) = make_float4(rv[0], rv[1], rv[2], rv[3]);
              }
            }
          }
        }
      }
    }
  }
  __syncthreads();  // O complete

  // h0^T = Wo^T . O^T + X_last
#pragma unroll
  for (int qi = 0; qi < QFW; ++qi) {
    const int qf = wave * QFW + qi;
    if (qf < NQF) {
      f32x4 acc[NMF];
#pragma unroll
      for (int nf = 0; nf < NMF; ++nf) acc[nf] = f32x4{0.f, 0.f, 0.f, 0.f};
      uint4 wo[2];
      wo[0] = a.Wo[qf * 64 + lane];
#pragma unroll
      for (int ks = 0; ks < KSTEPS; ++ks) {
        if (ks + 1 < KSTEPS) wo[(ks + 1) & 1] = a.Wo[((ks + 1) * NB + qf) * 64 + lane];
#pragma unroll
        for (int nf = 0; nf < NMF; ++nf) {
          const uint4 bo = *(const uint4*)(Xl + (nf * 16 + lc) * XLSTR + ks * 64 + lg * 16);
          M::run(acc[nf], wo[ks & 1], bo);
        }
      }
#pragma unroll
      for (int nf = 0; nf < NMF; ++nf) {
        const int m = nf * 16 + lc;
        const int64_t n = tile0 + m;
        if (n < N) {
          const int d = qf * 16 + 4 * lg;
          float4 r;
          if (a.Xin) {  // the residual: the input row itself (fp32)
            const float4 x = *reinterpret_cast<const float4*>(a.Xin + (n * T + T - 1) * D + d);
            r = make_float4(acc[nf][0] + x.x, acc[nf][1] + x.y, acc[nf][2] + x.z, acc[nf][3] + x.w);
          } else {
            const int j = (int)(((uint32_t)d * einv) >> 20), cc = d - j * a.e;
            const int byte = Wb[m * 64 + (T - 1) * a.g + j];
            r.x = acc[nf][0] + (M::val(E[byte * a.e + cc]) + M::val(P[(T - 1) * D + d]));
            r.y = acc[nf][1] + (M::val(E[byte * a.e + cc + 1]) + M::val(P[(T - 1) * D + d + 1]));
            r.z = acc[nf][2] + (M::val(E[byte * a.e + cc + 2]) + M::val(P[(T - 1) * D + d + 2]));
            r.w = acc[nf][3] + (M::val(E[byte * a.e + cc + 3]) + M::val(P[(T - 1) * D + d + 3]));
          }
          *reinterpret_cast<float4*>(a.h0 + n * D + d) = r;
        }
      }
    }
  }
}

// ------------------------------------------------- shared byte groups ----
// k_attn_grp: the same block for bf16 tiles of MA consecutive windows of one
// stream.  Windows at positions i and i + g share T-1 of their tokens (their
// bytes are grouped from the same alignment), and a token's projection is
// E.W + P.W with the positional part a table row, so the E-part of a byte
// group's q, K and V is computed once for all the windows that hold it.
// Wave w takes the NPW = MA/8 windows i = c + g*(b*NPW + i') of alignment class
// c = w % g (b = w / g): their NPW*T tokens are the NPW + T - 1 groups
// r = i' + t, one 16-row MFMA fragment.  Per head the wave writes its groups'
// K_h (then V_h) to its own LDS rows; lanes (i', t) form the scores
// q . (K_E[i'+t] + (P.Wk)[t]) and the softmax over t (aligned groups of T
// lanes), and lanes (i', 4 features) form sum_t a_t (V_E[i'+t] + (P.Wv)[t]).
template <int T, int G, int D, int DH>
struct GrpShape {
  static constexpr int NW = 8, MA = 64, NPW = MA / NW, W = T * G;
  static constexpr int KSTEPS = D / 32, NFH = DH / 16;
  static constexpr int KSC = (KSTEPS * NFH <= 16) ? KSTEPS : 16 / NFH;  // k-steps per staged 16 KiB chunk
  static constexpr int CHUNK = KSC * NFH * 64;
  // E_last / O rows: unpadded, 16-byte unit u of row m stored at u ^ (m & XXM)
  static constexpr int XLSTR = D * 2, XXM = (D / 8 >= 16 ? 16 : D / 8) - 1;
  static constexpr int KVSTR = DH + 4;  // floats per group row in the exchange (unpadded swizzled rows: slower)
  static constexpr int WB = MA + W + 64;
  // q and attention weights are stored class-major (a wave's windows in
  // consecutive rows) with padded rows, so a wave's reads hit distinct banks
  static constexpr int QSTR = D + 4, PSTR = T + 1;
  static constexpr int LDS = 2 * CHUNK * 16 + MA * QSTR * 4 + MA * XLSTR + WB + NW * 16 * KVSTR * 4 + MA * PSTR * 4 +
                             2 * 2 * T * DH * 4;
  static constexpr bool ok = (8 % G == 0) && NPW + T - 1 <= 16 && LDS <= 160 * 1024;
};

template <int T, int G, int D, int DH>
__global__ __launch_bounds__(512) void k_attn_grp(AttnArgs a) {
  typedef Mma<true> M;
  typedef GrpShape<T, G, D, DH> S;
  constexpr int H = D / DH, NW = S::NW, MA = S::MA, NPW = S::NPW, W = S::W;
  constexpr int KSTEPS = S::KSTEPS, NFH = S::NFH, KSC = S::KSC, CPP = KSTEPS / KSC, CHUNK = S::CHUNK;
  constexpr int XLSTR = S::XLSTR, KVSTR = S::KVSTR;
  constexpr int NQF = D / 16, QFW = (NQF + NW - 1) / NW, NMF = MA / 16, NB = D / 16;
  constexpr int WPD = 1;  // k-steps ahead that the q and output-projection weight fragments are fetched (3: no gain)
  constexpr int CQ = DH / 4;  // 4-feature chunks of a head
  static_assert(S::ok && KSTEPS % KSC == 0 && (T == 4 || T == 8), "shape");
  __shared__ uint4 Wst[2][CHUNK];
  constexpr int QSTR = S::QSTR, PSTR = S::PSTR;
  __shared__ __align__(16) float Qs[MA * QSTR];            // q, row cm(i) of window i
  __shared__ __align__(16) unsigned char Xl[MA * XLSTR];  // E_last rows, then O rows
  __shared__ __align__(16) float KV[NW][16 * KVSTR];       // this wave's group rows of K_h, then V_h
  __shared__ float Ps[MA * PSTR];                          // attention weights, row cm(i)
  __shared__ __align__(16) float PKV[2][2][T * DH];       // head slices of P.Wk and P.Wv, double-buffered
  __shared__ uint8_t Wb[S::WB];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, lg = lane >> 4, lc = lane & 15;
  const int64_t tile0 = (int64_t)blockIdx.x * MA;
  const int64_t N = a.w.N;
  const uint16_t* __restrict__ E = (const uint16_t*)a.E;
  const uint16_t* __restrict__ P = (const uint16_t*)a.P;
  const float* __restrict__ PQ = a.PW;
  const float* __restrict__ PK = a.PW + (int64_t)T * D;
  const float* __restrict__ PV = a.PW + (int64_t)2 * T * D;

  // the tile's bytes: Wb[k] = stream byte at (target of window 0) - W + k,
  // k < MA + W (all windows of the tile lie in one stream)
  {
    const int64_t base = target_offset(a.w, tile0) - W;
    for (int k = tid; k < S::WB; k += 512) Wb[k] = k < MA + W ? a.w.streams[base + k] : 0;
  }
  const uint32_t einv = ((1u << 20) + (uint32_t)a.e - 1u) / (uint32_t)a.e;
  const int cls = wave % G, blk = wave / G;
  // window (tile index) of this wave's i'-th window
  auto win_of = [&](int ip) { return cls + G * (blk * NPW + ip); };
  // class-major row of window i (the windows of a wave are consecutive rows)
  auto cm = [&](int i) { return ((i % G) + G * ((i / G) / NPW)) * NPW + (i / G) % NPW; };
  __syncthreads();

  // this wave's groups r = 0..15 as B fragments (E-part); the last group of each
  // window (r = i' + T - 1) also to LDS as that window's E_last row
  uint4 xb[KSTEPS];
  {
    const int r = lc;
    const int off = cls + G * (blk * NPW + r);  // first byte of group r in Wb
    const int ip = r - (T - 1);
    int byte[KSTEPS];
#pragma unroll
    for (int ks = 0; ks < KSTEPS; ++ks) {
      const int d = ks * 32 + lg * 8;
      const int j = (int)(((uint32_t)d * einv) >> 20);
      byte[ks] = Wb[off + j];
    }
#pragma unroll
    for (int ks = 0; ks < KSTEPS; ++ks) {
      const int d = ks * 32 + lg * 8;
      const int j = (int)(((uint32_t)d * einv) >> 20), cc = d - j * a.e;
      xb[ks] = *reinterpret_cast<const uint4*>(E + byte[ks] * a.e + cc);
    }
    if (ip >= 0 && ip < NPW) {
#pragma unroll
      for (int ks = 0; ks < KSTEPS; ++ks)
        *(uint4*)(Xl + win_of(ip) * XLSTR + 16 * ((ks * 4 + lg) ^ (win_of(ip) & S::XXM))) = xb[ks];
    }
  }
  __syncthreads();

  // fragment reads of Xl rows nf*16 + lc at units 4 ks + lg: byte 64 (ks & ~3) + xo[ks & 3]
  int xo[4];
  {
    const int q = (lc & S::XXM) >> 2, p = lg ^ (lc & 3);
#pragma unroll
    for (int j = 0; j < 4; ++j) xo[j] = 16 * (((j ^ q) << 2) | p);
  }
  // q^T = Wq^T . E_last^T + (P.Wq)[T-1] ; lane holds q[m = nf*16 + lc][c = qf*16 + 4*lg + r]
#pragma unroll
  for (int qi = 0; qi < QFW; ++qi) {
    const int qf = wave * QFW + qi;
    if (qf < NQF) {
      f32x4 acc[NMF];
#pragma unroll
      for (int nf = 0; nf < NMF; ++nf) acc[nf] = f32x4{0.f, 0.f, 0.f, 0.f};
      // weight fragments (L2) fetched WPD k-steps ahead
      uint4 wq[WPD + 1];
#pragma unroll
      for (int ks = 0; ks < WPD && ks < KSTEPS; ++ks) wq[ks] = a.Wq[(ks * NB + qf) * 64 + lane];
#pragma unroll
      for (int ks = 0; ks < KSTEPS; ++ks) {
        if (ks + WPD < KSTEPS) wq[(ks + WPD) % (WPD + 1)] = a.Wq[((ks + WPD) * NB + qf) * 64 + lane];
#pragma unroll
        for (int nf = 0; nf < NMF; ++nf) {
          const uint4 bx = *(const uint4*)(Xl + (nf * 16 + lc) * XLSTR + (ks & ~3) * 64 + xo[ks & 3]);
          M::run(acc[nf], wq[ks % (WPD + 1)], bx);
        }
      }
      const float4 pq = *reinterpret_cast<const float4*>(PQ + (T - 1) * D + qf * 16 + 4 * lg);
#pragma unroll
      for (int nf = 0; nf < NMF; ++nf) {
        const int m = nf * 16 + lc;
        *reinterpret_cast<float4*>(Qs + cm(m) * QSTR + qf * 16 + 4 * lg) =
            make_float4(acc[nf][0] + pq.x, acc[nf][1] + pq.y, acc[nf][2] + pq.z, acc[nf][3] + pq.w);
      }
    }
  }

  auto chunk_src = [&](int c, int i) -> const uint4* {
    const int ck = c % CPP, pass = (c / CPP) & 1, h = c / (2 * CPP);
    const int kk = i / (NFH * 64), f = (i / 64) % NFH, ln = i & 63;
    const uint4* Wp = pass ? a.Wv : a.Wk;
    return Wp + ((ck * KSC + kk) * NB + h * NFH + f) * 64 + ln;
  };
  constexpr int NFRAG = KSC * NFH;
  auto stage = [&](int c, int buf) {
#pragma unroll
    for (int q = wave; q < NFRAG; q += NW)
      __builtin_amdgcn_global_load_lds((const void*)chunk_src(c, q * 64 + lane),
                                       (__attribute__((address_space(3))) void*)(Wst[buf] + q * 64), 16, 0, 0);
  };
  constexpr int NCH = H * 2 * CPP;
  // rows t of P.Wk and P.Wv of head hh -> PKV[hh & 1] by direct 16-byte loads,
  // slot l = (which * T + t) * DH / 4 + c4 (T <= 8 <= DH / 4)
  constexpr int PKV_SLOTS = 2 * T * DH / 4;
  auto stage_pkv = [&](int hh) {
    if (wave * 64 < PKV_SLOTS) {
      const int l = wave * 64 + lane;
      const int which = l / (T * DH / 4), t = (l / (DH / 4)) % T, c4 = l % (DH / 4);
      // unit c4 of row t holds features 4 (c4 ^ t) .. + 3 (rows of different t read
      // at one unit hit different banks)
      const float* src = (which ? PV : PK) + t * D + hh * DH + 4 * (c4 ^ t);
      __builtin_amdgcn_global_load_lds((const void*)src,
                                       (__attribute__((address_space(3))) void*)(&PKV[hh & 1][0][0] + wave * 256), 16,
                                       0, 0);
    }
  };
  static_assert(PKV_SLOTS % 64 == 0 && T <= DH / 4, "PKV staging by whole waves; swizzle within a row");
  stage(0, 0);
  stage_pkv(0);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();  // chunk 0 and head 0's P rows staged; Qs complete; E_last rows no longer needed

  const float scale = a.scale;
  float* kv = KV[wave];
  const int row0 = wave * NPW;  // this wave's first class-major row (cm(win_of(0)))
  // lanes as (window i', token t) pairs for the scores
  const int sp_i = lane / T, sp_t = lane - (lane / T) * T;
  const bool sp_live = sp_i < NPW;
  for (int h = 0; h < H; ++h) {
    // this head's rows of P.Wk and P.Wv are in PKV[h & 1]: staged during the
    // previous head (head 0 with the first weight chunk)
    const float* pkh = PKV[h & 1][0];
    const float* pvh = PKV[h & 1][1];
#pragma unroll
    for (int pass = 0; pass < 2; ++pass) {
      f32x4 acc[NFH];
#pragma unroll
      for (int f = 0; f < NFH; ++f) acc[f] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ck = 0; ck < CPP; ++ck) {
        const int c = (h * 2 + pass) * CPP + ck;
        if (c + 1 < NCH) stage(c + 1, (c + 1) & 1);
        const uint4* buf = Wst[c & 1];
#pragma unroll
        for (int kk = 0; kk < KSC; ++kk) {
#pragma unroll
          for (int f = 0; f < NFH; ++f) M::run(acc[f], buf[(kk * NFH + f) * 64 + lane], xb[ck * KSC + kk]);
        }
        __builtin_amdgcn_s_waitcnt(0);
        __syncthreads();
        // every wave is past head h - 1, the last reader of PKV[(h + 1) & 1]:
        // stage head h + 1's P rows there (waited for at the next chunk barrier)
        if (pass == 0 && ck == 0 && h + 1 < H) stage_pkv(h + 1);
      }
      // group rows of K_h (E-part) or V_h to this wave's exchange rows
#pragma unroll
      for (int f = 0; f < NFH; ++f)
        *reinterpret_cast<float4*>(kv + lc * KVSTR + f * 16 + 4 * lg) =
            make_float4(acc[f][0], acc[f][1], acc[f][2], acc[f][3]);
      __builtin_amdgcn_wave_barrier();
      if (pass == 0) {
        float s = 0.f;
        if (sp_live) {
          const float* qv = Qs + (row0 + sp_i) * QSTR + h * DH;
          const float* kr = kv + (sp_i + sp_t) * KVSTR;
          const float* pk = pkh + sp_t * DH;
#pragma unroll
          for (int c4 = 0; c4 < CQ; ++c4) {
            const float4 q4 = *reinterpret_cast<const float4*>(qv + 4 * c4);
            const float4 k4 = *reinterpret_cast<const float4*>(kr + 4 * c4);
            const float4 p4 = *reinterpret_cast<const float4*>(pk + 4 * (c4 ^ sp_t));
            s += q4.x * (k4.x + p4.x) + q4.y * (k4.y + p4.y) + q4.z * (k4.z + p4.z) + q4.w * (k4.w + p4.w);
          }
        }
        s *= scale;
        const float mx = group_max<T>(s);
        const float pe = expf(s - mx);
        const float sm = group_sum<T>(pe);
        if (sp_live) Ps[(row0 + sp_i) * PSTR + sp_t] = pe * __builtin_amdgcn_rcpf(sm);
      } else {
        // O_h[i'][4 cq .. 4 cq + 3] = sum_t a_t (V_E[i'+t] + (P.Wv)[t]) -> O rows (bf16)
#pragma unroll
        for (int pr0 = 0; pr0 < NPW * CQ; pr0 += 64) {
          const int pr = pr0 + lane;
          if (pr < NPW * CQ) {
            const int ip = pr / CQ, cq = pr - (pr / CQ) * CQ;
            float4 o = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
            for (int t = 0; t < T; ++t) {
              const float at = Ps[(row0 + ip) * PSTR + t];
              const float4 v4 = *reinterpret_cast<const float4*>(kv + (ip + t) * KVSTR + 4 * cq);
              const float4 p4 = *reinterpret_cast<const float4*>(pvh + t * DH + 4 * (cq ^ t));
              o.x += at * (v4.x + p4.x);
              o.y += at * (v4.y + p4.y);
              o.z += at * (v4.z + p4.z);
              o.w += at * (v4.w + p4.w);
            }
            const int orow = win_of(ip), oe = h * DH + 4 * cq;
            put4o((uint16_t*)(Xl + orow * XLSTR + 16 * ((oe >> 3) ^ (orow & S::XXM)) + 8 * ((oe >> 2) & 1)),
                  f32x4{o.x, o.y, o.z, o.w});
          }
        }
      }
      __builtin_amdgcn_wave_barrier();
    }
  }
  __syncthreads();  // O complete; q no longer needed

  // h0^T = Wo^T . O^T + X_last (fp32: E + P of the last token), rows staged in
  // the q tile (padded rows: conflict-free), then written out whole
#pragma unroll
  for (int qi = 0; qi < QFW; ++qi) {
    const int qf = wave * QFW + qi;
    if (qf < NQF) {
      f32x4 acc[NMF];
#pragma unroll
      for (int nf = 0; nf < NMF; ++nf) acc[nf] = f32x4{0.f, 0.f, 0.f, 0.f};
      uint4 wo[WPD + 1];
#pragma unroll
      for (int ks = 0; ks < WPD && ks < KSTEPS; ++ks) wo[ks] = a.Wo[(ks * NB + qf) * 64 + lane];
#pragma unroll
      for (int ks = 0; ks < KSTEPS; ++ks) {
        if (ks + WPD < KSTEPS) wo[(ks + WPD) % (WPD + 1)] = a.Wo[((ks + WPD) * NB + qf) * 64 + lane];
#pragma unroll
        for (int nf = 0; nf < NMF; ++nf) {
          const uint4 bo = *(const uint4*)(Xl + (nf * 16 + lc) * XLSTR + (ks & ~3) * 64 + xo[ks & 3]);
          M::run(acc[nf], wo[ks % (WPD + 1)], bo);
        }
      }
#pragma unroll
      for (int nf = 0; nf < NMF; ++nf) {
        const int m = nf * 16 + lc;
        const int d = qf * 16 + 4 * lg;
        const int j = (int)(((uint32_t)d * einv) >> 20), cc = d - j * a.e;
        const int byte = Wb[m + (T - 1) * G + j];
        float4 r;
        r.x = acc[nf][0] + (M::val(E[byte * a.e + cc]) + M::val(P[(T - 1) * D + d]));
        r.y = acc[nf][1] + (M::val(E[byte * a.e + cc + 1]) + M::val(P[(T - 1) * D + d + 1]));
        r.z = acc[nf][2] + (M::val(E[byte * a.e + cc + 2]) + M::val(P[(T - 1) * D + d + 2]));
        r.w = acc[nf][3] + (M::val(E[byte * a.e + cc + 3]) + M::val(P[(T - 1) * D + d + 3]));
        *reinterpret_cast<float4*>(Qs + m * QSTR + d) = r;
      }
    }
  }
  __syncthreads();
  // the tile's h0 rows are one contiguous block of MA * D floats: each wave
  // writes whole rows, 16 bytes per lane
  for (int m = wave; m < MA; m += NW) {
    const int64_t n = tile0 + m;
    if (n < N) {
#pragma unroll
      for (int c = 4 * lane; c < D; c += 256)
        *reinterpret_cast<float4*>(a.h0 + n * D + c) = *reinterpret_cast<const float4*>(Qs + m * QSTR + c);
    }
  }
}

// ------------------------------------------------------- one head per wave ----
// k_attn_wh: the result of k_attn_grp for 64-window tiles of the shape with 8
// heads of 32 features, g = 8 and T = 4 or 8, with the work cut by head
// instead of by window.  Window i of the tile reads its token t from the group
// that starts i + g t bytes into the tile's bytes, so the tile holds
// MA + W - g distinct groups ("group rows" o); their E-parts go to LDS once
// (16-byte unit u of row o at u ^ (o & 15), conflict-free fragment reads).
// Wave h then forms everything of head h with no barrier until the output
// projection:
//   K_h^T = Wk_h^T . X_E^T over all group rows, q_h^T = Wq_h^T . E_last^T +
//     (P.Wq)[T-1] (E_last of window i is group row i + g (T-1));
//   a lane's accumulator quads hold group row 16 rf + lc (K) and window
//     16 nf + lc (q), features 4 lg + r of each 16-feature block.  Key row
//     i + g t of window 16 nf + lc is row lc of fragment nf + t/2 for even t;
//     for odd t it is row lc ^ 8 of fragment nf + (t-1)/2 + (lc >= 8): each
//     lane picks the fragment its partner needs and a DPP rotation by 8 lanes
//     within the row of 16 brings it over (once per fragment, shift8);
//   scores q . (K_E[row] + (P.Wk)[t]) as partial sums over the lane's 8
//     features, summed over the 4 lane groups by a reduce-scatter (shuffles
//     across 32 and 16 lanes) that leaves lane (lg, lc) with the T scores of
//     window 16 lg + lc: softmax in the lane; the weights go through this
//     wave's LDS rows to the lanes that hold each window;
//   V_h^T = Wv_h^T . X_E^T and O_h = sum_t a_t (V_E[row] + (P.Wv)[t]) with the
//     same row selection, rounded to bf16 into the O tile.
// The output projection and residual follow as in k_attn_grp, the waves split
// over output features.
template <int T, int G, int D, int DH>
struct WhShape {
  static constexpr int NW = 8, MA = 64, W = T * G, H = D / DH;
  static constexpr int NRF = (MA + W - G + 15) / 16;  // group-row fragments
  static constexpr int NWF = MA / 16;                  // window fragments
  static constexpr int KSTEPS = D / 32, NB = D / 16;
  static constexpr int XSTR = D * 2, XM = (D / 8 >= 16 ? 16 : D / 8) - 1;
  static constexpr int HSTR = D + 4;  // h0 rows staged for the write (floats, padded)
  static constexpr int XG = NRF * 16 * XSTR > MA * HSTR * 4 ? NRF * 16 * XSTR : MA * HSTR * 4;
  static constexpr int WB = MA + W + 64;
  static constexpr int LDS = XG + MA * XSTR + 2 * T * D * 4 + NW * MA * T * 4 + WB;
  static constexpr bool ok = H == NW && DH == 32 && G == 8 && (T == 4 || T == 8) && D == 256 &&
                             (NRF * 16 * (D / 8)) % 512 == 0 && LDS <= 160 * 1024;
};

// x from lane lc ^ 8 of the same row of 16 lanes
__device__ __forceinline__ float ror8(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x128, 0xF, 0xF, false));
}

// The group rows 8 below each fragment's: sh[j] lane lc holds row
// 16 j + lc + 8, taken from fragment j (lc < 8) or j + 1 (lc >= 8) of the
// partner lane lc ^ 8.  Row i + G t of window i = 16 nf + lc is then
// acc[nf + t/2] for even t and sh[nf + (t-1)/2] for odd t.
template <int NRF, int NSH>
__device__ __forceinline__ void shift8(const f32x4 (&acc)[NRF][2], f32x4 (&sh)[NSH][2], bool hi) {
  static_assert(NSH < NRF, "rows");
#pragma unroll
  for (int j = 0; j < NSH; ++j)
#pragma unroll
    for (int fr = 0; fr < 2; ++fr)
#pragma unroll
      for (int r = 0; r < 4; ++r) sh[j][fr][r] = ror8(hi ? acc[j][fr][r] : acc[j + 1][fr][r]);
}
template <int NRF, int NSH>
__device__ __forceinline__ const f32x4& key_row(const f32x4 (&acc)[NRF][2], const f32x4 (&sh)[NSH][2], int nf, int t,
                                                int fr) {
  return (t & 1) == 0 ? acc[nf + t / 2][fr] : sh[nf + t / 2][fr];
}

template <int T, int G, int D, int DH>
__global__ __launch_bounds__(512) void k_attn_wh(AttnArgs a) {
  typedef Mma<true> M;
  typedef WhShape<T, G, D, DH> S;
  constexpr int NW = S::NW, MA = S::MA, W = S::W, NRF = S::NRF, NWF = S::NWF, KSTEPS = S::KSTEPS, NB = S::NB;
  constexpr int XSTR = S::XSTR, XM = S::XM, HSTR = S::HSTR;
  constexpr int EPB = D / G;            // features per byte embedding
  constexpr int QOFF = (T - 1) * G;     // group row of window 0's last token
  constexpr int NQF = D / 16, QFW = NQF / NW;
  static_assert(S::ok, "shape");
  __shared__ __align__(16) unsigned char Xg[S::XG];      // group rows (bf16), later the h0 rows (fp32)
  __shared__ __align__(16) unsigned char Xo[MA * XSTR];  // O rows (bf16)
  __shared__ __align__(16) float PKV[2][T * D];          // P.Wk, P.Wv
  __shared__ __align__(16) float Aw[NW][MA * T];         // each wave's attention weights, one row per window
  __shared__ uint8_t Wb[S::WB];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, lg = lane >> 4, lc = lane & 15;
  const int h = wave;
  const int64_t tile0 = (int64_t)blockIdx.x * MA;
  const int64_t N = a.w.N;
  const uint16_t* __restrict__ E = (const uint16_t*)a.E;
  const uint16_t* __restrict__ P = (const uint16_t*)a.P;

  // the tile's bytes: Wb[k] = stream byte at (target of window 0) - W + k
  {
    const int64_t base = target_offset(a.w, tile0) - W;
    for (int k = tid; k < S::WB; k += 512) Wb[k] = k < MA + W ? a.w.streams[base + k] : 0;
    const float4* src = reinterpret_cast<const float4*>(a.PW + (int64_t)T * D);
    for (int k = tid; k < 2 * T * D / 4; k += 512) reinterpret_cast<float4*>(&PKV[0][0])[k] = src[k];
  }
  __syncthreads();
  // group rows o: unit u holds features 8u .. 8u + 7, from byte o + u / (EPB / 8)
  {
    constexpr int NU = NRF * 16 * (D / 8) / 512;
    uint4 ev[NU];
#pragma unroll
    for (int r = 0; r < NU; ++r) {
      const int q = tid + 512 * r, o = q / (D / 8), u = q % (D / 8);
      const int byte = Wb[o + u / (EPB / 8)];
      ev[r] = *reinterpret_cast<const uint4*>(E + byte * EPB + (u % (EPB / 8)) * 8);
    }
#pragma unroll
    for (int r = 0; r < NU; ++r) {
      const int q = tid + 512 * r, o = q / (D / 8), u = q % (D / 8);
      *(uint4*)(Xg + o * XSTR + 16 * (u ^ (o & XM))) = ev[r];
    }
  }
  __syncthreads();

  // fragment reads of rows m (m & 15 = c) at units 4 ks + lg: byte 64 (ks & ~3) + off[ks & 3]
  auto swz = [&](int c, int (&off)[4]) {
    const int q = (c & XM) >> 2, p = lg ^ (c & 3);
#pragma unroll
    for (int j = 0; j < 4; ++j) off[j] = 16 * (((j ^ q) << 2) | p);
  };
  int xo[4], qo[4];
  swz(lc, xo);
  swz((QOFF + lc) & 15, qo);
  const bool hi = lc >= 8;

  // K_h over all group rows and q_h over the windows' last tokens
  f32x4 kacc[NRF][2], qacc[NWF][2];
#pragma unroll
  for (int rf = 0; rf < NRF; ++rf) kacc[rf][0] = kacc[rf][1] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int nf = 0; nf < NWF; ++nf) qacc[nf][0] = qacc[nf][1] = f32x4{0.f, 0.f, 0.f, 0.f};
  {
    const uint4* Wkh = a.Wk + (h * 2) * 64 + lane;
    const uint4* Wqh = a.Wq + (h * 2) * 64 + lane;
    uint4 wk[2][2], wq[2][2];
#pragma unroll
    for (int fr = 0; fr < 2; ++fr) {
      wk[0][fr] = Wkh[fr * 64];
      wq[0][fr] = Wqh[fr * 64];
    }
#pragma unroll
    for (int ks = 0; ks < KSTEPS; ++ks) {
      if (ks + 1 < KSTEPS) {
#pragma unroll
        for (int fr = 0; fr < 2; ++fr) {
          wk[(ks + 1) & 1][fr] = Wkh[((ks + 1) * NB + fr) * 64];
          wq[(ks + 1) & 1][fr] = Wqh[((ks + 1) * NB + fr) * 64];
        }
      }
      const int kb = (ks & ~3) * 64;
      uint4 bg[NRF], bq[NWF];
#pragma unroll
      for (int rf = 0; rf < NRF; ++rf) bg[rf] = *(const uint4*)(Xg + (16 * rf + lc) * XSTR + kb + xo[ks & 3]);
#pragma unroll
      for (int nf = 0; nf < NWF; ++nf) bq[nf] = *(const uint4*)(Xg + (QOFF + 16 * nf + lc) * XSTR + kb + qo[ks & 3]);
#pragma unroll
      for (int rf = 0; rf < NRF; ++rf)
#pragma unroll
        for (int fr = 0; fr < 2; ++fr) M::run(kacc[rf][fr], wk[ks & 1][fr], bg[rf]);
#pragma unroll
      for (int nf = 0; nf < NWF; ++nf)
#pragma unroll
        for (int fr = 0; fr < 2; ++fr) M::run(qacc[nf][fr], wq[ks & 1][fr], bq[nf]);
    }
  }
  {
    const float* pq = a.PW + (T - 1) * D + h * DH + 4 * lg;
#pragma unroll
    for (int fr = 0; fr < 2; ++fr) {
      const float4 p4 = *reinterpret_cast<const float4*>(pq + 16 * fr);
#pragma unroll
      for (int nf = 0; nf < NWF; ++nf) {
        qacc[nf][fr][0] += p4.x;
        qacc[nf][fr][1] += p4.y;
        qacc[nf][fr][2] += p4.z;
        qacc[nf][fr][3] += p4.w;
      }
    }
  }

  // scores: partial sums over the lane's 8 features
  constexpr int NSH = NWF + (T - 1) / 2;
  float sc[NWF][T];
  {
    f32x4 ksh[NSH][2];
    shift8(kacc, ksh, hi);
    const float* pk = &PKV[0][0] + h * DH + 4 * lg;
#pragma unroll
    for (int t = 0; t < T; ++t) {
      const float4 p0 = *reinterpret_cast<const float4*>(pk + t * D);
      const float4 p1 = *reinterpret_cast<const float4*>(pk + t * D + 16);
#pragma unroll
      for (int nf = 0; nf < NWF; ++nf) {
        const f32x4& k0 = key_row(kacc, ksh, nf, t, 0);
        const f32x4& k1 = key_row(kacc, ksh, nf, t, 1);
        const f32x4& q0 = qacc[nf][0];
        const f32x4& q1 = qacc[nf][1];
        float s = q0[0] * (k0[0] + p0.x) + q0[1] * (k0[1] + p0.y) + q0[2] * (k0[2] + p0.z) + q0[3] * (k0[3] + p0.w);
        s += q1[0] * (k1[0] + p1.x) + q1[1] * (k1[1] + p1.y) + q1[2] * (k1[2] + p1.z) + q1[3] * (k1[3] + p1.w);
        sc[nf][t] = s;
      }
    }
  }
  // reduce-scatter over the lane groups: lane (lg, lc) ends with window 16 lg + lc
  float st[T];
  {
    const bool up = lg >= 2, od = (lg & 1) != 0;
    float r1[2][T];
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int t = 0; t < T; ++t) {
        const float keep = up ? sc[2 + j][t] : sc[j][t];
        const float send = up ? sc[j][t] : sc[2 + j][t];
        r1[j][t] = keep + __shfl_xor(send, 32, 64);
      }
#pragma unroll
    for (int t = 0; t < T; ++t) {
      const float keep = od ? r1[1][t] : r1[0][t];
      const float send = od ? r1[0][t] : r1[1][t];
      st[t] = keep + __shfl_xor(send, 16, 64);
    }
  }
  {
    const float scale = a.scale;
    float mx = -INFINITY;
#pragma unroll
    for (int t = 0; t < T; ++t) {
      st[t] *= scale;
      mx = fmaxf(mx, st[t]);
    }
    float sm = 0.f;
#pragma unroll
    for (int t = 0; t < T; ++t) {
      st[t] = expf(st[t] - mx);
      sm += st[t];
    }
    const float rs = __builtin_amdgcn_rcpf(sm);
    float* aw = Aw[wave] + (16 * lg + lc) * T;
#pragma unroll
    for (int t = 0; t < T; t += 4)
      *reinterpret_cast<float4*>(aw + t) = make_float4(st[t] * rs, st[t + 1] * rs, st[t + 2] * rs, st[t + 3] * rs);
  }

  // V_h over all group rows
  f32x4 vacc[NRF][2];
#pragma unroll
  for (int rf = 0; rf < NRF; ++rf) vacc[rf][0] = vacc[rf][1] = f32x4{0.f, 0.f, 0.f, 0.f};
  {
    const uint4* Wvh = a.Wv + (h * 2) * 64 + lane;
    uint4 wv[2][2];
#pragma unroll
    for (int fr = 0; fr < 2; ++fr) wv[0][fr] = Wvh[fr * 64];
#pragma unroll
    for (int ks = 0; ks < KSTEPS; ++ks) {
      if (ks + 1 < KSTEPS) {
#pragma unroll
        for (int fr = 0; fr < 2; ++fr) wv[(ks + 1) & 1][fr] = Wvh[((ks + 1) * NB + fr) * 64];
      }
      const int kb = (ks & ~3) * 64;
      uint4 bg[NRF];
#pragma unroll
      for (int rf = 0; rf < NRF; ++rf) bg[rf] = *(const uint4*)(Xg + (16 * rf + lc) * XSTR + kb + xo[ks & 3]);
#pragma unroll
      for (int rf = 0; rf < NRF; ++rf)
#pragma unroll
        for (int fr = 0; fr < 2; ++fr) M::run(vacc[rf][fr], wv[ks & 1][fr], bg[rf]);
    }
  }
  __builtin_amdgcn_wave_barrier();
  // O_h[window 16 nf + lc][features 16 fr + 4 lg + r]
  {
    float aa[NWF][T];
#pragma unroll
    for (int nf = 0; nf < NWF; ++nf) {
      const float* aw = Aw[wave] + (16 * nf + lc) * T;
#pragma unroll
      for (int t = 0; t < T; t += 4) {
        const float4 v = *reinterpret_cast<const float4*>(aw + t);
        aa[nf][t] = v.x;
        aa[nf][t + 1] = v.y;
        aa[nf][t + 2] = v.z;
        aa[nf][t + 3] = v.w;
      }
    }
    f32x4 vsh[NSH][2];
    shift8(vacc, vsh, hi);
    f32x4 o[NWF][2];
#pragma unroll
    for (int nf = 0; nf < NWF; ++nf) o[nf][0] = o[nf][1] = f32x4{0.f, 0.f, 0.f, 0.f};
    const float* pv = &PKV[1][0] + h * DH + 4 * lg;
#pragma unroll
    for (int t = 0; t < T; ++t) {
      const float4 p0 = *reinterpret_cast<const float4*>(pv + t * D);
      const float4 p1 = *reinterpret_cast<const float4*>(pv + t * D + 16);
#pragma unroll
      for (int nf = 0; nf < NWF; ++nf) {
        const f32x4& v0 = key_row(vacc, vsh, nf, t, 0);
        const f32x4& v1 = key_row(vacc, vsh, nf, t, 1);
        const float at = aa[nf][t];
        o[nf][0][0] += at * (v0[0] + p0.x);
        o[nf][0][1] += at * (v0[1] + p0.y);
        o[nf][0][2] += at * (v0[2] + p0.z);
        o[nf][0][3] += at * (v0[3] + p0.w);
        o[nf][1][0] += at * (v1[0] + p1.x);
        o[nf][1][1] += at * (v1[1] + p1.y);
        o[nf][1][2] += at * (v1[2] + p1.z);
        o[nf][1][3] += at * (v1[3] + p1.w);
      }
    }
#pragma unroll
    for (int nf = 0; nf < NWF; ++nf) {
      const int m = 16 * nf + lc;
#pragma unroll
      for (int fr = 0; fr < 2; ++fr) {
        const int oe = h * DH + 16 * fr + 4 * lg;
        put4o((uint16_t*)(Xo + m * XSTR + 16 * ((oe >> 3) ^ (m & XM)) + 8 * ((oe >> 2) & 1)), o[nf][fr]);
      }
    }
  }
  __syncthreads();  // O complete; group rows no longer needed

  // h0^T = Wo^T . O^T + X_last (fp32: E + P of the last token), rows staged
  // over the group rows, then written out whole
  float* Hs = reinterpret_cast<float*>(Xg);
#pragma unroll
  for (int qi = 0; qi < QFW; ++qi) {
    const int qf = wave * QFW + qi;
    f32x4 acc[NWF];
#pragma unroll
    for (int nf = 0; nf < NWF; ++nf) acc[nf] = f32x4{0.f, 0.f, 0.f, 0.f};
    uint4 wo[2];
    wo[0] = a.Wo[qf * 64 + lane];
#pragma unroll
    for (int ks = 0; ks < KSTEPS; ++ks) {
      if (ks + 1 < KSTEPS) wo[(ks + 1) & 1] = a.Wo[((ks + 1) * NB + qf) * 64 + lane];
#pragma unroll
      for (int nf = 0; nf < NWF; ++nf) {
        const uint4 bo = *(const uint4*)(Xo + (16 * nf + lc) * XSTR + (ks & ~3) * 64 + xo[ks & 3]);
        M::run(acc[nf], wo[ks & 1], bo);
      }
    }
#pragma unroll
    for (int nf = 0; nf < NWF; ++nf) {
      const int m = 16 * nf + lc;
      const int d = qf * 16 + 4 * lg;
      const int j = d / EPB, cc = d - j * EPB;
      const int byte = Wb[m + QOFF + j];
      float4 r;
      r.x = acc[nf][0] + (M::val(E[byte * EPB + cc]) + M::val(P[(T - 1) * D + d]));
      r.y = acc[nf][1] + (M::val(E[byte * EPB + cc + 1]) + M::val(P[(T - 1) * D + d + 1]));
      r.z = acc[nf][2] + (M::val(E[byte * EPB + cc + 2]) + M::val(P[(T - 1) * D + d + 2]));
      r.w = acc[nf][3] + (M::val(E[byte * EPB + cc + 3]) + M::val(P[(T - 1) * D + d + 3]));
      *reinterpret_cast<float4*>(Hs + m * HSTR + d) = r;
    }
  }
  __syncthreads();
  for (int m = wave; m < MA; m += NW) {
    const int64_t n = tile0 + m;
    if (n < N) {
#pragma unroll
      for (int c = 4 * lane; c < D; c += 256)
        *reinterpret_cast<float4*>(a.h0 + n * D + c) = *reinterpret_cast<const float4*>(Hs + m * HSTR + c);
    }
  }
}

// ------------------------------------------------------------ dispatch ----
// Measured alternative, slower on the main workload (2^20 windows): two
// accumulator sets so that the scores of head h run under the MFMAs of its V
// pass and its weighted sum under those of the next K pass: 3.4 ms against 3.2.
template <bool BF, int T, int D, int DH, bool SMALL>
static void launch_attn(const AttnArgs& a, hipStream_t s) {
  typedef AttnShape<BF, T, D, DH, SMALL> S;
  static_assert(S::LDS <= 160 * 1024, "LDS");
  const dim3 grid((unsigned)((a.w.N + S::MA - 1) / S::MA));
  if (a.Om) {
    if (a.kK)
      hipLaunchKernelGGL((k_attn<BF, T, D, DH, true, SMALL, true>), grid, dim3(512), 0, s, a);
    else
      hipLaunchKernelGGL((k_attn<BF, T, D, DH, false, SMALL, true>), grid, dim3(512), 0, s, a);
  } else if (a.kK) {
    hipLaunchKernelGGL((k_attn<BF, T, D, DH, true, SMALL, false>), grid, dim3(512), 0, s, a);
  } else {
    hipLaunchKernelGGL((k_attn<BF, T, D, DH, false, SMALL, false>), grid, dim3(512), 0, s, a);
  }
}

template <int T, int G, int D, int DH>
static bool launch_grp(const AttnArgs& a, hipStream_t s) {
  if constexpr (WhShape<T, G, D, DH>::ok) {
    hipLaunchKernelGGL((k_attn_wh<T, G, D, DH>), dim3((unsigned)((a.w.N + 63) / 64)), dim3(512), 0, s, a);
    return true;
  } else if constexpr (GrpShape<T, G, D, DH>::ok) {
    hipLaunchKernelGGL((k_attn_grp<T, G, D, DH>), dim3((unsigned)((a.w.N + 63) / 64)), dim3(512), 0, s, a);
    return true;
  }
  return false;
}

// bf16 launches whose 64-window tiles each lie in one stream (steps per stream
// and the launch's first window multiples of 64) share the byte groups
// (k_attn_grp) unless the caller asks for the per-token kernel, whose result
// for a window does not depend on the launch; launches too small to give every CU a workgroup at the widest
// token tile (one step of the update path) take one 16-row fragment per wave.
template <bool BF, int T, int D, int DH>
static void run_attn(const AttnArgs& a, hipStream_t s) {
  if constexpr (BF) {
    if (!a.kK && !a.token_only && a.w.n_steps % 64 == 0 && a.w.n0 % 64 == 0) {
      if (a.g == 8 && launch_grp<T, 8, D, DH>(a, s)) return;
      if (a.g == 4 && launch_grp<T, 4, D, DH>(a, s)) return;
    }
  }
  if (a.w.N >= (int64_t)256 * AttnShape<BF, T, D, DH>::MA || AttnShape<BF, T, D, DH>::RFW == 1)
    launch_attn<BF, T, D, DH, false>(a, s);
  else
    launch_attn<BF, T, D, DH, true>(a, s);
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
