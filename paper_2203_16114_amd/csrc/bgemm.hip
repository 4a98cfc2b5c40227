// GEMM of the update step on bf16 MFMAs (Alg. 1: the backward of the
// estimator's loss, every product of which is a plain matrix product).
//
// Operands are read as fp32 straight from where the update step keeps them,
// in either orientation: k contiguous (activation gradients times weights,
// dY . W^T) or m / n contiguous (weight gradients, act^T . dY).  Each thread
// reads its share of the next 128 x 64 k-tile with float4 loads while the
// current tile is multiplied, converts it in registers (one v_cvt_pk_bf16_f32
// per pair, round to nearest even) and writes whole 16-byte units of 8 k
// values to LDS, in an XOR-swizzled layout whose fragment reads are free of
// bank conflicts.  Operands that are fp32 values rather than bf16 storage
// points are split into hi = bf16(v) and lo = bf16(v - hi) (v - hi is exact in
// fp32), and their products take two MFMAs (hi.B + lo.B), which keeps about
// 16 significant bits of v.  A product may have two K segments summed into
// one result (C = A1.B1 + A2.B2, as the two halves of the input gradient of
// the key and value projections), so that C is written once.
// Split-K partial sums go to a workspace and are added in a fixed order, so
// results do not depend on scheduling.  Blocks are ordered so that the tiles
// that share operand rows run on one XCD (one L2).
#include <type_traits>

#include "kcommon.h"
#include "kernels.h"

namespace {

constexpr int BM = 128, BN = 128, BK = 64;
constexpr int UNITS = BM * BK * 2 / 16;  // 16-byte units per 128 x 64 bf16 tile (1024)

inline int64_t rup(int64_t x, int64_t a) { return (x + a - 1) / a * a; }

typedef float f32x2v __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2v __attribute__((ext_vector_type(2)));

// (a, b) -> bf16 pair, a in the low half, each rounded to nearest even
__device__ __forceinline__ uint32_t pk_bf(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2v{a, b}, bf16x2v));
}
// bf16 pair of the residuals (a - hi_a, b - hi_b), h = pk_bf(a, b)
__device__ __forceinline__ uint32_t pk_lo(float a, float b, uint32_t h) {
  return pk_bf(a - __uint_as_float(h << 16), b - __uint_as_float(h & 0xffff0000u));
}
__device__ __forceinline__ float comp(const float4& v, int i) {
  return i == 0 ? v.x : (i == 1 ? v.y : (i == 2 ? v.z : v.w));
}

// One operand: up to two K segments, element (row, k) of segment s at
// p_s[row * ld_s + k] (k contiguous) or p_s[k * ld_s + row].  Segment 1 starts
// at k = k1p of the product (segment 0's extent rounded up to BK).  (Named
// fields, not arrays: an array indexed at run time would live in scratch.)
struct Src {
  const float* p0;
  const float* p1;
  int64_t ld0, ld1;
  int kext0, kext1;
  int k1p;
  int rows;
  // rank-one rows (GemmArgs::r1c; one segment, rows contiguous, fp32):
  // element (k, n) = (r1c[(w H + n >> dsh) << tsh | t] . V(w, n)) . r1scale, k = w << tsh | t
  const float* r1c;
  int r1tsh, r1dsh, r1H, r1round;
  float r1scale;
};

// Element of a rank-one source at k (absolute within the segment) and
// column n (its head n >> dsh): (c . V(w, n)) r1scale, V(w, n) = x.
__device__ __forceinline__ float r1v(const Src& s, int k, int n, float x) {
  const int w = k >> s.r1tsh, t = k & ((1 << s.r1tsh) - 1);
  const float c = s.r1c[(((int64_t)w * s.r1H + (n >> s.r1dsh)) << s.r1tsh) + t];
  if (s.r1round) x = __uint_as_float(pack_bf16x2(x, 0.f) << 16);
  return (c * x) * s.r1scale;
}
// The eight coefficients c of k = k0 .. k0 + 7, k0 a multiple of 8, T = 8:
// one window w = k0 / 8, t = 0 .. 7, head n >> dsh (two 16-byte loads).
__device__ __forceinline__ void r1c8(const Src& s, int k0, int n, float (&c)[8]) {
  const float* p = s.r1c + (((int64_t)(k0 >> 3) * s.r1H + (n >> s.r1dsh)) << 3);
  const float4 a = *reinterpret_cast<const float4*>(p), b = *reinterpret_cast<const float4*>(p + 4);
  c[0] = a.x; c[1] = a.y; c[2] = a.z; c[3] = a.w;
  c[4] = b.x; c[5] = b.y; c[6] = b.z; c[7] = b.w;
}
__device__ __forceinline__ float r1round(const Src& s, float x) {
  return s.r1round ? __uint_as_float(pack_bf16x2(x, 0.f) << 16) : x;
}

// LDS unit (16 bytes) of (row, k-chunk c) in a swizzled 128 x 64 tile: the
// chunk XOR-ed with (row ^ row >> 2) & 7, measured free of bank conflicts both
// for the 16-row fragment reads and for the unit writes of operands whose rows
// are contiguous (with row & 7 alone those writes were 8-way conflicted).
__device__ __forceinline__ int unit_of(int row, int c) { return row * 8 + (c ^ ((row ^ (row >> 2)) & 7)); }

// This thread's 32 values of the 128 x 64 tile (rows row0.., k k0..).  k
// contiguous: units u = tid + 256 q (row u / 8, chunk u % 8), two float4 each.
// Rows contiguous: rows 4 (tid % 32) .. +3 of chunk tid / 32, one float4 per k
// (lanes along the rows, for coalesced loads).
// Every load is made, from an address clamped into the operand; bit j of the
// returned mask says whether float4 j lies inside, and store_tile zeroes the
// others.  (A load under a condition is compiled into a load from a select of
// the address and a zero in scratch memory, and a select right after the load
// would wait for it before the multiply.)
// H: the operand is stored as bf16 (pointer and strides in bf16 elements).  k
// contiguous: one 16-byte unit of 8 k values per (row, chunk), its bits in
// v[2q] (the operand's K is a multiple of 8; bits 2q, 2q+1 of the mask both say
// whether the unit lies inside).  Rows contiguous: per k, the 8 bytes of rows
// 4 (tid % 32) .. +3 as the bits of v[j].x, v[j].y.
template <bool KC, bool H>
__device__ __forceinline__ uint32_t load_tile_h(const Src& s, int row0, int k0, int tid, float4 (&v)[8]) {
  const bool seg1 = k0 >= s.k1p;
  const uint16_t* __restrict__ p = (const uint16_t*)(seg1 ? s.p1 : s.p0);
  const int ld = (int)(seg1 ? s.ld1 : s.ld0);
  const int kk0 = seg1 ? k0 - s.k1p : k0, kr = (seg1 ? s.kext1 : s.kext0) - kk0;
  uint32_t mask = 0;
  auto at = [](const uint16_t* base, int off) { return reinterpret_cast<const char*>(base) + (uint32_t)off * 2u; };
  if constexpr (KC) {
    const uint16_t* base = p + (int64_t)row0 * ld + kk0;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int u = tid + 256 * q, rr = u >> 3, c8 = (u & 7) * 8;
      const int ro = min(rr, s.rows - 1 - row0) * ld;
      v[2 * q] = __builtin_bit_cast(float4, *reinterpret_cast<const uint4*>(at(base, ro + min(c8, kr - 8))));
      v[2 * q + 1] = make_float4(0.f, 0.f, 0.f, 0.f);
      const uint32_t in = (row0 + rr < s.rows && c8 < kr) ? 3u : 0u;
      mask |= in << (2 * q);
    }
  } else {
    const uint16_t* base = p + (int64_t)kk0 * ld + row0;
    const int rr = 4 * (tid & 31), kc = (tid >> 5) * 8;
    const bool rin = row0 + rr < s.rows;
    const int ro = min(rr, s.rows - 4 - row0);
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const uint2 w = *reinterpret_cast<const uint2*>(at(base, min(kc + j, kr - 1) * ld + ro));
      v[j] = make_float4(__uint_as_float(w.x), __uint_as_float(w.y), 0.f, 0.f);
      mask |= (uint32_t)(rin && kc + j < kr) << j;
    }
  }
  return mask;
}

template <bool KC, bool H = false>
__device__ __forceinline__ uint32_t load_tile(const Src& s, int row0, int k0, int tid, float4 (&v)[8]) {
  if constexpr (H) return load_tile_h<KC, true>(s, row0, k0, tid, v);
  const bool seg1 = k0 >= s.k1p;
  const float* __restrict__ p = seg1 ? s.p1 : s.p0;
  const int ld = (int)(seg1 ? s.ld1 : s.ld0);
  const int kk0 = seg1 ? k0 - s.k1p : k0, kr = (seg1 ? s.kext1 : s.kext0) - kk0;  // k values left
  uint32_t mask = 0;
  // per-tile base in scalar registers, 32-bit offsets within the tile
  auto ld4 = [](const float* base, int off) {
    return *reinterpret_cast<const float4*>(reinterpret_cast<const char*>(base) + (uint32_t)off * 4u);
  };
  if constexpr (KC) {
    const float* base = p + (int64_t)row0 * ld + kk0;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int u = tid + 256 * q, rr = u >> 3, c8 = (u & 7) * 8;
      const int ro = min(rr, s.rows - 1 - row0) * ld;
      v[2 * q] = ld4(base, ro + min(c8, kr - 4));
      v[2 * q + 1] = ld4(base, ro + min(c8 + 4, kr - 4));
      const bool rin = row0 + rr < s.rows;
      mask |= (uint32_t)(rin && c8 < kr) << (2 * q);
      mask |= (uint32_t)(rin && c8 + 4 < kr) << (2 * q + 1);
    }
  } else {
    const float* base = p + (int64_t)kk0 * ld + row0;
    const int rr = 4 * (tid & 31), kc = (tid >> 5) * 8;
    const bool rin = row0 + rr < s.rows;
    const int ro = min(rr, s.rows - 4 - row0);
    if (s.r1c) {  // rows of V: window k >> tsh
      const int n = row0 + ro;
      if (s.r1tsh == 3 && kc + 8 <= kr) {  // the eight k of one window: V(w, n..n+3) once
        const int k0 = kk0 + kc;
        float4 x = *reinterpret_cast<const float4*>(p + (int64_t)(k0 >> 3) * ld + n);
        x = make_float4(r1round(s, x.x), r1round(s, x.y), r1round(s, x.z), r1round(s, x.w));
        float c[8];
        r1c8(s, k0, n, c);
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          v[j] = make_float4((c[j] * x.x) * s.r1scale, (c[j] * x.y) * s.r1scale, (c[j] * x.z) * s.r1scale,
                             (c[j] * x.w) * s.r1scale);
          mask |= (uint32_t)rin << j;
        }
        return mask;
      }
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int k = kk0 + min(kc + j, kr - 1);
        const float4 x = *reinterpret_cast<const float4*>(p + (int64_t)(k >> s.r1tsh) * ld + n);
        v[j] = make_float4(r1v(s, k, n, x.x), r1v(s, k, n, x.y), r1v(s, k, n, x.z), r1v(s, k, n, x.w));
        mask |= (uint32_t)(rin && kc + j < kr) << j;
      }
      return mask;
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      v[j] = ld4(base, min(kc + j, kr - 1) * ld + ro);
      mask |= (uint32_t)(rin && kc + j < kr) << j;
    }
  }
  return mask;
}

// The values of load_tile (float4 j zero unless bit j of mask) -> bf16 units
// of the LDS tile hi (and lo when split).
// bf16 pairs (k, k + 1) of one row from two words that each hold two rows:
// the low halves (row 0 of the pair) or the high halves (row 1)
__device__ __forceinline__ uint32_t pair_lo(uint32_t wa, uint32_t wb) { return __builtin_amdgcn_perm(wb, wa, 0x05040100u); }
__device__ __forceinline__ uint32_t pair_hi(uint32_t wa, uint32_t wb) { return __builtin_amdgcn_perm(wb, wa, 0x07060302u); }

template <bool KC, bool SPLIT, bool H = false>
__device__ __forceinline__ void store_tile(const float4 (&vin)[8], uint32_t mask, uint4* hi, uint4* lo, int tid) {
  if constexpr (H) {  // bf16 source: the units as loaded (k contiguous) or packed per row
    static_assert(!SPLIT, "a bf16 operand is not split");
    if constexpr (KC) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int u = tid + 256 * q;
        const uint32_t m = 0u - ((mask >> (2 * q)) & 1u);
        const uint4 w = __builtin_bit_cast(uint4, vin[2 * q]);
        hi[unit_of(u >> 3, u & 7)] = make_uint4(w.x & m, w.y & m, w.z & m, w.w & m);
      }
    } else {
      const int rr = 4 * (tid & 31), c = tid >> 5;
      uint32_t w[8][2];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const uint32_t m = 0u - ((mask >> j) & 1u);
        w[j][0] = __float_as_uint(vin[j].x) & m;
        w[j][1] = __float_as_uint(vin[j].y) & m;
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        uint32_t x[4];
#pragma unroll
        for (int pp = 0; pp < 4; ++pp)
          x[pp] = (i & 1) ? pair_hi(w[2 * pp][i >> 1], w[2 * pp + 1][i >> 1])
                          : pair_lo(w[2 * pp][i >> 1], w[2 * pp + 1][i >> 1]);
        hi[unit_of(rr + i, c)] = make_uint4(x[0], x[1], x[2], x[3]);
      }
    }
    return;
  }
  float4 v[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const uint32_t m = 0u - ((mask >> j) & 1u);
    v[j] = make_float4(__uint_as_float(__float_as_uint(vin[j].x) & m), __uint_as_float(__float_as_uint(vin[j].y) & m),
                       __uint_as_float(__float_as_uint(vin[j].z) & m), __uint_as_float(__float_as_uint(vin[j].w) & m));
  }
  if constexpr (KC) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int u = tid + 256 * q, at = unit_of(u >> 3, u & 7);
      const float4 a = v[2 * q], b = v[2 * q + 1];
      const uint4 h = make_uint4(pk_bf(a.x, a.y), pk_bf(a.z, a.w), pk_bf(b.x, b.y), pk_bf(b.z, b.w));
      hi[at] = h;
      if constexpr (SPLIT)
        lo[at] = make_uint4(pk_lo(a.x, a.y, h.x), pk_lo(a.z, a.w, h.y), pk_lo(b.x, b.y, h.z), pk_lo(b.z, b.w, h.w));
    }
  } else {
    const int rr = 4 * (tid & 31), c = tid >> 5;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int at = unit_of(rr + i, c);
      float x[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) x[j] = comp(v[j], i);
      const uint4 h = make_uint4(pk_bf(x[0], x[1]), pk_bf(x[2], x[3]), pk_bf(x[4], x[5]), pk_bf(x[6], x[7]));
      hi[at] = h;
      if constexpr (SPLIT)
        lo[at] = make_uint4(pk_lo(x[0], x[1], h.x), pk_lo(x[2], x[3], h.y), pk_lo(x[4], x[5], h.z),
                            pk_lo(x[6], x[7], h.w));
    }
  }
}

// C[m][n] (+)= sum_k A(m, k) B(k, n) over this split's k range.  AKC / BKC:
// that operand's contiguous dimension is k; SA / SB: that operand is split.
// 1-D grid of tn * tm * splits blocks.
template <bool AKC, bool BKC, bool SA, bool SB, bool HA, bool HB>
__global__ __launch_bounds__(256) void k_bgemm(Src A, Src B, int Kp, int M, int N, float* C, int64_t ldc,
                                               float beta, float* __restrict__ part, int kchunk, int tn, int tm,
                                               const float* __restrict__ gu, int hc, const float* cin) {
  static_assert(!(SA && SB), "at most one operand is split");
  constexpr int NT = 2 + (SA ? 1 : 0) + (SB ? 1 : 0);  // tiles per stage: A hi, B hi, [A lo | B lo]
  __shared__ uint4 lds[2][NT][UNITS];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, lg = lane >> 4, lc = lane & 15;
  const int wm = wave >> 1, wn = wave & 1;
  // workgroups go to the 8 XCDs in turn: give each XCD a run of consecutive
  // tiles (n fastest), which share rows of A and k ranges of B
  const int nb = (int)gridDim.x, b = (int)blockIdx.x, per = nb / 8;
  const int L = b < per * 8 ? (b & 7) * per + (b >> 3) : b;
  const int bx = L % tn, by = (L / tn) % tm, bz = L / (tn * tm);
  const int m0 = by * BM, n0 = bx * BN;
  const int kb = bz * kchunk, ke = min(Kp, kb + kchunk);
  f32x4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  float4 va[8], vb[8];
  uint32_t ma = 0, mb_ = 0;
  auto put = [&](int buf) {
    store_tile<AKC, SA, HA>(va, ma, lds[buf][0], lds[buf][SA ? 2 : 0], tid);
    store_tile<BKC, SB, HB>(vb, mb_, lds[buf][1], lds[buf][NT - 1], tid);
  };
  if (kb < ke) {
    ma = load_tile<AKC, HA>(A, m0, kb, tid, va);
    mb_ = load_tile<BKC, HB>(B, n0, kb, tid, vb);
    put(0);
  }
  __syncthreads();
  int buf = 0;
  for (int k0 = kb; k0 < ke; k0 += BK, buf ^= 1) {
    const bool more = k0 + BK < ke;
    if (more) {  // next tile into registers while this one is multiplied
      ma = load_tile<AKC, HA>(A, m0, k0 + BK, tid, va);
      mb_ = load_tile<BKC, HB>(B, n0, k0 + BK, tid, vb);
    }
    // keep the order loads / multiply / LDS writes: otherwise the writes to the
    // other buffer are hoisted above the multiply and wait on the loads at once
    asm volatile("" ::: "memory");
#pragma unroll
    for (int ks = 0; ks < BK / 32; ++ks) {
      const int c = ks * 4 + lg;
      uint4 af[4], bf[4];
#pragma unroll
      for (int rf = 0; rf < 4; ++rf) af[rf] = lds[buf][0][unit_of(wm * 64 + rf * 16 + lc, c)];
#pragma unroll
      for (int nf = 0; nf < 4; ++nf) bf[nf] = lds[buf][1][unit_of(wn * 64 + nf * 16 + lc, c)];
#pragma unroll
      for (int rf = 0; rf < 4; ++rf)
#pragma unroll
        for (int nf = 0; nf < 4; ++nf) Mma<true>::run(acc[rf][nf], af[rf], bf[nf]);
      if constexpr (SA) {
#pragma unroll
        for (int rf = 0; rf < 4; ++rf) af[rf] = lds[buf][2][unit_of(wm * 64 + rf * 16 + lc, c)];
#pragma unroll
        for (int rf = 0; rf < 4; ++rf)
#pragma unroll
          for (int nf = 0; nf < 4; ++nf) Mma<true>::run(acc[rf][nf], af[rf], bf[nf]);
      }
      if constexpr (SB) {  // (SA and SB are never both set: af still holds A hi)
#pragma unroll
        for (int nf = 0; nf < 4; ++nf) bf[nf] = lds[buf][NT - 1][unit_of(wn * 64 + nf * 16 + lc, c)];
#pragma unroll
        for (int rf = 0; rf < 4; ++rf)
#pragma unroll
          for (int nf = 0; nf < 4; ++nf) Mma<true>::run(acc[rf][nf], af[rf], bf[nf]);
      }
    }
    asm volatile("" ::: "memory");
    // the other buffer was last read before the previous barrier
    if (more) put(buf ^ 1);
    __syncthreads();
  }
  // lane holds C[m0 + wm*64 + rf*16 + 4*lg + r][n0 + wn*64 + nf*16 + lc]
  const int mb = m0 + wm * 64 + 4 * lg, nbase = n0 + wn * 64 + lc;
  if (part) {
    float* pz = part + (int64_t)bz * M * N;
#pragma unroll
    for (int rf = 0; rf < 4; ++rf)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = mb + rf * 16 + r;
        if (m >= M) continue;
#pragma unroll
        for (int nf = 0; nf < 4; ++nf) {
          const int n = nbase + nf * 16;
          if (n < N) pz[(int64_t)m * N + n] = acc[rf][nf][r];
        }
      }
  } else {
    // with beta = 1, all the values of Cin (which may be C) are read before any
    // C is written
    if (beta != 0.f) {  // clamped addresses, as for gu below
#pragma unroll
      for (int rf = 0; rf < 4; ++rf) {
        float c[4][4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int64_t mo = (int64_t)min(mb + rf * 16 + r, M - 1) * ldc;
#pragma unroll
          for (int nf = 0; nf < 4; ++nf) c[r][nf] = cin[mo + min(nbase + nf * 16, N - 1)];
        }
#pragma unroll
        for (int r = 0; r < 4; ++r)
#pragma unroll
          for (int nf = 0; nf < 4; ++nf) acc[rf][nf][r] += c[r][nf];
      }
    }
    if (gu) {  // C = (A.B) * GELU'(U), U laid out as C
      // loads from clamped addresses, all of a fragment row before any use
      // (elements outside C are computed but not stored); U is read once,
      // streamed past the caches (large workload's update 0.884 -> 0.873 ms)
#pragma unroll
      for (int rf = 0; rf < 4; ++rf) {
        float u[4][4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int64_t mo = (int64_t)min(mb + rf * 16 + r, M - 1) * ldc;
#pragma unroll
          for (int nf = 0; nf < 4; ++nf) u[r][nf] = __builtin_nontemporal_load(gu + mo + min(nbase + nf * 16, N - 1));
        }
#pragma unroll
        for (int r = 0; r < 4; ++r)
#pragma unroll
          for (int nf = 0; nf < 4; ++nf) acc[rf][nf][r] *= gelu_grad_as(u[r][nf]);
      }
    }
#pragma unroll
    for (int rf = 0; rf < 4; ++rf)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = mb + rf * 16 + r;
        if (m >= M) continue;
#pragma unroll
        for (int nf = 0; nf < 4; ++nf) {
          const int n = nbase + nf * 16;
          if (n < N) {
            if (hc)
              reinterpret_cast<uint16_t*>(C)[(int64_t)m * ldc + n] = f2bf(acc[rf][nf][r]);
            else
              C[(int64_t)m * ldc + n] = acc[rf][nf][r];
          }
        }
      }
  }
}

// ---- 256 x 256 tiles, 512 threads (8 waves, two per SIMD), 32 k per stage ----
// Twice the MFMA work per operand byte read of the 128 x 128 kernel, for the
// large products.  Each wave owns a 64 x 128 block of C when A is split (its
// rows are read twice from LDS, hi and lo) and a 128 x 64 block otherwise.
namespace big {
constexpr int TM = 256, TN = 256, TK = 32;
constexpr int UNITS = TM * TK * 2 / 16;  // 16-byte units per 256 x 32 bf16 tile (1024)

// LDS unit of (row, k-chunk c): 4 units per row, the chunk swizzled by bits
// 1..2 of the row (16-row fragment reads measured free of bank conflicts;
// bits 2..3 were 2-way conflicted).
__device__ __forceinline__ int unit_of(int row, int c) { return row * 4 + (c ^ ((row >> 1) & 3)); }

// This thread's 16 values of the 256 x 32 tile (rows row0.., k k0..).  k
// contiguous: units u = tid + 512 q (row u / 4, chunk u % 4), two float4
// each.  Rows contiguous: rows 2 (tid % 128), +1 of chunk tid / 128, a float2
// per k (v[j / 2] holds k = 2 (j / 2), +1).  Same clamping and mask as
// load_tile.
// H: bf16 source.  k contiguous: unit q (8 k) bits in v[2q], mask bits 2q and
// 2q + 1 both set when it lies inside.  Rows contiguous: per k the 4 bytes of
// rows 2 (tid % 128), +1, k = 2i, 2i + 1 in v[i].x, v[i].y.
template <bool KC>
__device__ __forceinline__ uint32_t load_h(const Src& s, int row0, int k0, int tid, float4 (&v)[4]) {
  const bool seg1 = k0 >= s.k1p;
  const uint16_t* __restrict__ p = (const uint16_t*)(seg1 ? s.p1 : s.p0);
  const int ld = (int)(seg1 ? s.ld1 : s.ld0);
  const int kk0 = seg1 ? k0 - s.k1p : k0, kr = (seg1 ? s.kext1 : s.kext0) - kk0;
  uint32_t mask = 0;
  auto at = [](const uint16_t* base, int off) { return reinterpret_cast<const char*>(base) + (uint32_t)off * 2u; };
  if constexpr (KC) {
    const uint16_t* base = p + (int64_t)row0 * ld + kk0;
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const int u = tid + 512 * q, rr = u >> 2, c8 = (u & 3) * 8;
      const int ro = min(rr, s.rows - 1 - row0) * ld;
      v[2 * q] = __builtin_bit_cast(float4, *reinterpret_cast<const uint4*>(at(base, ro + min(c8, kr - 8))));
      v[2 * q + 1] = make_float4(0.f, 0.f, 0.f, 0.f);
      const uint32_t in = (row0 + rr < s.rows && c8 < kr) ? 3u : 0u;
      mask |= in << (2 * q);
    }
  } else {
    const uint16_t* base = p + (int64_t)kk0 * ld + row0;
    const int rr = 2 * (tid & 127), kc = (tid >> 7) * 8;
    const bool rin = row0 + rr < s.rows;
    const int ro = min(rr, s.rows - 2 - row0);
#pragma unroll
    for (int j = 0; j < 8; j += 2) {
      const uint32_t a = *reinterpret_cast<const uint32_t*>(at(base, min(kc + j, kr - 1) * ld + ro));
      const uint32_t b = *reinterpret_cast<const uint32_t*>(at(base, min(kc + j + 1, kr - 1) * ld + ro));
      v[j >> 1] = make_float4(__uint_as_float(a), __uint_as_float(b), 0.f, 0.f);
      mask |= (uint32_t)(rin && kc + j < kr) << j;
      mask |= (uint32_t)(rin && kc + j + 1 < kr) << (j + 1);
    }
  }
  return mask;
}

template <bool KC, bool H = false>
__device__ __forceinline__ uint32_t load(const Src& s, int row0, int k0, int tid, float4 (&v)[4]) {
  if constexpr (H) return load_h<KC>(s, row0, k0, tid, v);
  const bool seg1 = k0 >= s.k1p;
  const float* __restrict__ p = seg1 ? s.p1 : s.p0;
  const int ld = (int)(seg1 ? s.ld1 : s.ld0);
  const int kk0 = seg1 ? k0 - s.k1p : k0, kr = (seg1 ? s.kext1 : s.kext0) - kk0;
  uint32_t mask = 0;
  auto at = [](const float* base, int off) { return reinterpret_cast<const char*>(base) + (uint32_t)off * 4u; };
  if constexpr (KC) {
    const float* base = p + (int64_t)row0 * ld + kk0;
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const int u = tid + 512 * q, rr = u >> 2, c8 = (u & 3) * 8;
      const int ro = min(rr, s.rows - 1 - row0) * ld;
      v[2 * q] = *reinterpret_cast<const float4*>(at(base, ro + min(c8, kr - 4)));
      v[2 * q + 1] = *reinterpret_cast<const float4*>(at(base, ro + min(c8 + 4, kr - 4)));
      const bool rin = row0 + rr < s.rows;
      mask |= (uint32_t)(rin && c8 < kr) << (2 * q);
      mask |= (uint32_t)(rin && c8 + 4 < kr) << (2 * q + 1);
    }
  } else {
    const float* base = p + (int64_t)kk0 * ld + row0;
    const int rr = 2 * (tid & 127), kc = (tid >> 7) * 8;
    const bool rin = row0 + rr < s.rows;
    const int ro = min(rr, s.rows - 2 - row0);
    if (s.r1c) {  // rows of V: window k >> tsh
      const int n = row0 + ro;
      if (s.r1tsh == 3 && kc + 8 <= kr) {  // the eight k of one window: V(w, n..n+1) once
        const int k0 = kk0 + kc;
        float2 x = *reinterpret_cast<const float2*>(p + (int64_t)(k0 >> 3) * ld + n);
        x = make_float2(r1round(s, x.x), r1round(s, x.y));
        float c[8];
        r1c8(s, k0, n, c);
#pragma unroll
        for (int j = 0; j < 8; j += 2) {
          v[j >> 1] = make_float4((c[j] * x.x) * s.r1scale, (c[j] * x.y) * s.r1scale, (c[j + 1] * x.x) * s.r1scale,
                                  (c[j + 1] * x.y) * s.r1scale);
          mask |= (uint32_t)rin << j;
          mask |= (uint32_t)rin << (j + 1);
        }
        return mask;
      }
#pragma unroll
      for (int j = 0; j < 8; j += 2) {
        const int ka = kk0 + min(kc + j, kr - 1), kb = kk0 + min(kc + j + 1, kr - 1);
        const float2 a = *reinterpret_cast<const float2*>(p + (int64_t)(ka >> s.r1tsh) * ld + n);
        const float2 b = *reinterpret_cast<const float2*>(p + (int64_t)(kb >> s.r1tsh) * ld + n);
        v[j >> 1] = make_float4(r1v(s, ka, n, a.x), r1v(s, ka, n, a.y), r1v(s, kb, n, b.x), r1v(s, kb, n, b.y));
        mask |= (uint32_t)(rin && kc + j < kr) << j;
        mask |= (uint32_t)(rin && kc + j + 1 < kr) << (j + 1);
      }
      return mask;
    }
#pragma unroll
    for (int j = 0; j < 8; j += 2) {
      const float2 a = *reinterpret_cast<const float2*>(at(base, min(kc + j, kr - 1) * ld + ro));
      const float2 b = *reinterpret_cast<const float2*>(at(base, min(kc + j + 1, kr - 1) * ld + ro));
      v[j >> 1] = make_float4(a.x, a.y, b.x, b.y);
      mask |= (uint32_t)(rin && kc + j < kr) << j;
      mask |= (uint32_t)(rin && kc + j + 1 < kr) << (j + 1);
    }
  }
  return mask;
}

template <bool KC, bool SPLIT, bool H = false>
__device__ __forceinline__ void store(const float4 (&v)[4], uint32_t mask, uint4* hi, uint4* lo, int tid) {
  if constexpr (H) {
    static_assert(!SPLIT, "a bf16 operand is not split");
    if constexpr (KC) {
#pragma unroll
      for (int q = 0; q < 2; ++q) {
        const int u = tid + 512 * q;
        const uint32_t m = 0u - ((mask >> (2 * q)) & 1u);
        const uint4 w = __builtin_bit_cast(uint4, v[2 * q]);
        hi[unit_of(u >> 2, u & 3)] = make_uint4(w.x & m, w.y & m, w.z & m, w.w & m);
      }
    } else {
      const int rr = 2 * (tid & 127), c = tid >> 7;
      uint32_t w[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) w[j] = __float_as_uint((j & 1) ? v[j >> 1].y : v[j >> 1].x) & (0u - ((mask >> j) & 1u));
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        uint32_t x[4];
#pragma unroll
        for (int pp = 0; pp < 4; ++pp) x[pp] = i ? pair_hi(w[2 * pp], w[2 * pp + 1]) : pair_lo(w[2 * pp], w[2 * pp + 1]);
        hi[unit_of(rr + i, c)] = make_uint4(x[0], x[1], x[2], x[3]);
      }
    }
    return;
  }
  if constexpr (KC) {
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const int u = tid + 512 * q, at = unit_of(u >> 2, u & 3);
      const uint32_t m0 = 0u - ((mask >> (2 * q)) & 1u), m1 = 0u - ((mask >> (2 * q + 1)) & 1u);
      float x[8] = {v[2 * q].x, v[2 * q].y, v[2 * q].z, v[2 * q].w,
                    v[2 * q + 1].x, v[2 * q + 1].y, v[2 * q + 1].z, v[2 * q + 1].w};
#pragma unroll
      for (int j = 0; j < 8; ++j) x[j] = __uint_as_float(__float_as_uint(x[j]) & (j < 4 ? m0 : m1));
      const uint4 h = make_uint4(pk_bf(x[0], x[1]), pk_bf(x[2], x[3]), pk_bf(x[4], x[5]), pk_bf(x[6], x[7]));
      hi[at] = h;
      if constexpr (SPLIT)
        lo[at] = make_uint4(pk_lo(x[0], x[1], h.x), pk_lo(x[2], x[3], h.y), pk_lo(x[4], x[5], h.z),
                            pk_lo(x[6], x[7], h.w));
    }
  } else {
    const int rr = 2 * (tid & 127), c = tid >> 7;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int at = unit_of(rr + i, c);
      float x[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const float4& w = v[j >> 1];
        const float val = (j & 1) ? (i ? w.w : w.z) : (i ? w.y : w.x);
        x[j] = __uint_as_float(__float_as_uint(val) & (0u - ((mask >> j) & 1u)));
      }
      const uint4 h = make_uint4(pk_bf(x[0], x[1]), pk_bf(x[2], x[3]), pk_bf(x[4], x[5]), pk_bf(x[6], x[7]));
      hi[at] = h;
      if constexpr (SPLIT)
        lo[at] = make_uint4(pk_lo(x[0], x[1], h.x), pk_lo(x[2], x[3], h.y), pk_lo(x[4], x[5], h.z),
                            pk_lo(x[6], x[7], h.w));
    }
  }
}

// PD: stages whose loads are in flight while a stage is multiplied (1 or 2).
// With 2, the loads of stage s + 2 are issued before the multiply of stage s,
// and stage s + 1 (loaded during stage s - 1) goes to LDS after it: two stages
// of matrix work cover each load's latency (two register sets: operands read
// as bf16, or fp32 on one side only).
template <bool AKC, bool BKC, bool SA, bool SB, bool HA, bool HB, int PD>
__global__ __launch_bounds__(512) void k_bgemm_big(Src A, Src B, int Kp, int M, int N, float* C, int64_t ldc,
                                                   float beta, float* __restrict__ part, int kchunk, int tn, int tm,
                                                   const float* __restrict__ gu, int hc, const float* cin) {
  static_assert(!(SA && SB), "at most one operand is split");
  static_assert(PD == 1 || PD == 2, "prefetch depth");
  constexpr int NT = 2 + (SA ? 1 : 0) + (SB ? 1 : 0);
  constexpr int FM = SA ? 4 : 8, FN = SA ? 8 : 4;  // 16 x 16 fragments per wave along m, n
  constexpr int WN = TN / (16 * FN);                // waves along n
  __shared__ uint4 lds[2][NT][UNITS];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, lg = lane >> 4, lc = lane & 15;
  const int wm = wave / WN, wn = wave % WN;
  const int nb = (int)gridDim.x, b = (int)blockIdx.x, per = nb / 8;
  const int L = b < per * 8 ? (b & 7) * per + (b >> 3) : b;
  const int bx = L % tn, by = (L / tn) % tm, bz = L / (tn * tm);
  const int m0 = by * TM, n0 = bx * TN;
  const int kb = bz * kchunk, ke = min(Kp, kb + kchunk);
  f32x4 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  float4 va[PD][4], vb[PD][4];
  uint32_t ma[PD] = {}, mbk[PD] = {};
  auto ld = [&](int set, int k0) {
    ma[set] = load<AKC, HA>(A, m0, k0, tid, va[set]);
    mbk[set] = load<BKC, HB>(B, n0, k0, tid, vb[set]);
  };
  auto put = [&](int set, int buf) {
    store<AKC, SA, HA>(va[set], ma[set], lds[buf][0], lds[buf][SA ? 2 : 0], tid);
    store<BKC, SB, HB>(vb[set], mbk[set], lds[buf][1], lds[buf][NT - 1], tid);
  };
  auto mult = [&](int buf) {
    uint4 af[FM], bf[FN];
#pragma unroll
    for (int rf = 0; rf < FM; ++rf) af[rf] = lds[buf][0][unit_of(wm * 16 * FM + rf * 16 + lc, lg)];
#pragma unroll
    for (int nf = 0; nf < FN; ++nf) bf[nf] = lds[buf][1][unit_of(wn * 16 * FN + nf * 16 + lc, lg)];
#pragma unroll
    for (int rf = 0; rf < FM; ++rf)
#pragma unroll
      for (int nf = 0; nf < FN; ++nf) Mma<true>::run(acc[rf][nf], af[rf], bf[nf]);
    if constexpr (SA) {
#pragma unroll
      for (int rf = 0; rf < FM; ++rf) af[rf] = lds[buf][2][unit_of(wm * 16 * FM + rf * 16 + lc, lg)];
#pragma unroll
      for (int rf = 0; rf < FM; ++rf)
#pragma unroll
        for (int nf = 0; nf < FN; ++nf) Mma<true>::run(acc[rf][nf], af[rf], bf[nf]);
    }
    if constexpr (SB) {
#pragma unroll
      for (int nf = 0; nf < FN; ++nf) bf[nf] = lds[buf][NT - 1][unit_of(wn * 16 * FN + nf * 16 + lc, lg)];
#pragma unroll
      for (int rf = 0; rf < FM; ++rf)
#pragma unroll
        for (int nf = 0; nf < FN; ++nf) Mma<true>::run(acc[rf][nf], af[rf], bf[nf]);
    }
  };
  if constexpr (PD == 1) {
    if (kb < ke) {
      ld(0, kb);
      put(0, 0);
    }
    __syncthreads();
    int buf = 0;
    for (int k0 = kb; k0 < ke; k0 += TK, buf ^= 1) {
      const bool more = k0 + TK < ke;
      if (more) ld(0, k0 + TK);  // next tile into registers while this one is multiplied
      // keep the order loads / multiply / LDS writes: otherwise the writes to the
      // other buffer are hoisted above the multiply and wait on the loads at once
      asm volatile("" ::: "memory");
      mult(buf);
      asm volatile("" ::: "memory");
      if (more) put(0, buf ^ 1);  // the other buffer was last read before the previous barrier
      __syncthreads();
    }
  } else {
    // stage s (k = kb + s TK) in LDS buffer s & 1 and register set s & 1
    const int ns = (ke - kb + TK - 1) / TK;
    if (ns > 0) {
      ld(0, kb);
      put(0, 0);
    }
    if (ns > 1) ld(1, kb + TK);
    __syncthreads();
    // one stage: loads of s + 2 into its set (free: stage s went to LDS), the
    // multiply of s, and stage s + 1 (loaded a stage ago) from the other set to
    // the other buffer (last read before the previous barrier), its conversion
    // interleaved with the MFMAs.  The last stage writes that buffer too (a set
    // already stored, or never loaded): nothing reads it afterwards.
    constexpr int NMF = FM * FN * (1 + (SA ? 1 : 0) + (SB ? 1 : 0));
    auto stage = [&](auto cc, int st) {
      constexpr int c = decltype(cc)::value;
      if (st + 2 < ns) ld(c, kb + (st + 2) * TK);
      asm volatile("" ::: "memory");
      mult(c);
      put(c ^ 1, c ^ 1);
      __builtin_amdgcn_sched_group_barrier(0x100, FM + FN, 0);  // the first fragments
#pragma unroll
      for (int i = 0; i < NMF; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x002, 4, 0);
        if (i % 4 == 3) __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);
      }
      __syncthreads();
    };
    for (int st = 0; st < ns; st += 2) {
      stage(std::integral_constant<int, 0>{}, st);
      if (st + 1 < ns) stage(std::integral_constant<int, 1>{}, st + 1);
    }
  }
  const int mb = m0 + wm * 16 * FM + 4 * lg, nbase = n0 + wn * 16 * FN + lc;
  if (part) {
    float* pz = part + (int64_t)bz * M * N;
#pragma unroll
    for (int rf = 0; rf < FM; ++rf)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = mb + rf * 16 + r;
        if (m >= M) continue;
#pragma unroll
        for (int nf = 0; nf < FN; ++nf) {
          const int n = nbase + nf * 16;
          if (n < N) pz[(int64_t)m * N + n] = acc[rf][nf][r];
        }
      }
  } else {
    if (beta != 0.f) {  // clamped addresses, as for gu below
#pragma unroll
      for (int rf = 0; rf < FM; ++rf) {
        float c[4][FN];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int64_t mo = (int64_t)min(mb + rf * 16 + r, M - 1) * ldc;
#pragma unroll
          for (int nf = 0; nf < FN; ++nf) c[r][nf] = cin[mo + min(nbase + nf * 16, N - 1)];
        }
#pragma unroll
        for (int r = 0; r < 4; ++r)
#pragma unroll
          for (int nf = 0; nf < FN; ++nf) acc[rf][nf][r] += c[r][nf];
      }
    }
    if (gu) {  // C = (A.B) * GELU'(U), U laid out as C
      // loads from clamped addresses, all of a fragment row before any use
      // (elements outside C are computed but not stored); U is read once,
      // streamed past the caches (large workload's update 0.884 -> 0.873 ms)
#pragma unroll
      for (int rf = 0; rf < FM; ++rf) {
        float u[4][FN];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int64_t mo = (int64_t)min(mb + rf * 16 + r, M - 1) * ldc;
#pragma unroll
          for (int nf = 0; nf < FN; ++nf) u[r][nf] = __builtin_nontemporal_load(gu + mo + min(nbase + nf * 16, N - 1));
        }
#pragma unroll
        for (int r = 0; r < 4; ++r)
#pragma unroll
          for (int nf = 0; nf < FN; ++nf) acc[rf][nf][r] *= gelu_grad_as(u[r][nf]);
      }
    }
#pragma unroll
    for (int rf = 0; rf < FM; ++rf)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = mb + rf * 16 + r;
        if (m >= M) continue;
#pragma unroll
        for (int nf = 0; nf < FN; ++nf) {
          const int n = nbase + nf * 16;
          if (n < N) {
            if (hc)
              reinterpret_cast<uint16_t*>(C)[(int64_t)m * ldc + n] = f2bf(acc[rf][nf][r]);
            else
              C[(int64_t)m * ldc + n] = acc[rf][nf][r];
          }
        }
      }
  }
}

// split count of the 256-tile kernel (one block per CU): about 256 blocks,
// each split keeping at least 1024 k values; 0 when the product cannot fill
// the chip that way (shorter splits measured slower than the 128-tile kernel)
int splits(int M, int N, int Kp) {
  const int tiles = (int)(rup(M, TM) / TM * (rup(N, TN) / TN));
  int s = 1;
  while (tiles * s < 256 && Kp / (s * 2) >= 1024) s *= 2;
  return tiles * s >= 256 ? s : 0;
}

// PD = 2 where both register sets fit: an operand read as bf16 (its 16 values
// of a stage in 8 registers) and at most one fp32 operand
template <bool AKC, bool BKC>
void launch_orient(bool sa, bool sb, bool ha, bool hb, dim3 grid, const Src& A, const Src& B, int Kp, const GemmArgs& g,
                   float* part, int kchunk, int tn, int tm, hipStream_t s) {
#define TRACE_BGEMM(SA_, SB_, HA_, HB_, PD_)                                                                 \
  hipLaunchKernelGGL((k_bgemm_big<AKC, BKC, SA_, SB_, HA_, HB_, PD_>), grid, dim3(512), 0, s, A, B, Kp, g.M, g.N, g.C, \
                     g.ldc, g.beta, part, kchunk, tn, tm, g.gelu_u, g.halfC, g.Cin ? g.Cin : g.C)
  if (sa) {
    if (hb)
      TRACE_BGEMM(true, false, false, true, 2);
    else
      TRACE_BGEMM(true, false, false, false, 1);
  } else if (sb) {
    if (ha)
      TRACE_BGEMM(false, true, true, false, 2);
    else
      TRACE_BGEMM(false, true, false, false, 1);
  } else if (ha && hb) {
    TRACE_BGEMM(false, false, true, true, 2);
  } else if (ha) {
    TRACE_BGEMM(false, false, true, false, 2);
  } else if (hb) {
    TRACE_BGEMM(false, false, false, true, 2);
  } else {
    TRACE_BGEMM(false, false, false, false, 1);
  }
#undef TRACE_BGEMM
}
}  // namespace big

int bgemm_splits(int M, int N, int Kp) {
  const int tiles = (int)(rup(M, BM) / BM * (rup(N, BN) / BN));
  int splits = 1;
  // fill the 256 CUs about twice, each split keeping at least 512 k values
  // (shorter splits cost more in partial sums than they gain in parallelism)
  while (tiles * splits < 512 && Kp / (splits * 2) >= 512) splits *= 2;
  // products with few output tiles (weight gradients of narrow layers): fill
  // the CUs once with splits down to 256 k values
  while (tiles * splits < 256 && Kp / (splits * 2) >= 256) splits *= 2;
  return splits;
}

bool al16(const void* p) { return ((uintptr_t)p & 15) == 0; }

// Operand (rows x K, element (row, k) at p[row*srow + k*sk]; bf16 elements
// when half) as segment seg of src; false when the kernel's vector reads do not
// fit it (fp32: float4 along the contiguous dimension; bf16: 16-byte units of 8 k
// when k is contiguous, 8 bytes of 4 rows per k otherwise).
bool add_segment(Src& src, int seg, const float* p, int64_t srow, int64_t sk, int rows, int K, bool& kc, bool half) {
  const bool this_kc = sk == 1;
  if (!(this_kc || srow == 1)) return false;
  const int64_t ld = this_kc ? srow : sk;
  if (half) {
    if (this_kc ? (!al16(p) || ld % 8 != 0 || K % 8 != 0) : (((uintptr_t)p & 7) != 0 || ld % 4 != 0 || rows % 4 != 0))
      return false;
  } else if (!al16(p) || ld % 4 != 0 || (this_kc ? K % 4 : rows % 4) != 0) {
    return false;
  }
  if (ld > (1 << 20)) return false;  // byte offsets within a 128 x 64 tile stay below 2^31
  if (seg == 1 && this_kc != kc) return false;
  kc = this_kc;
  (seg ? src.p1 : src.p0) = p;
  (seg ? src.ld1 : src.ld0) = ld;
  (seg ? src.kext1 : src.kext0) = K;
  src.rows = rows;
  return true;
}

template <bool AKC, bool BKC>
void launch_orient(bool sa, bool sb, bool ha, bool hb, dim3 grid, const Src& A, const Src& B, int Kp, const GemmArgs& g,
                   float* part, int kchunk, int tn, int tm, hipStream_t s) {
#define TRACE_BGEMM(SA_, SB_, HA_, HB_)                                                                       \
  hipLaunchKernelGGL((k_bgemm<AKC, BKC, SA_, SB_, HA_, HB_>), grid, dim3(256), 0, s, A, B, Kp, g.M, g.N, g.C, g.ldc, \
                     g.beta, part, kchunk, tn, tm, g.gelu_u, g.halfC, g.Cin ? g.Cin : g.C)
  if (sa) {
    if (hb)
      TRACE_BGEMM(true, false, false, true);
    else
      TRACE_BGEMM(true, false, false, false);
  } else if (sb) {
    if (ha)
      TRACE_BGEMM(false, true, true, false);
    else
      TRACE_BGEMM(false, true, false, false);
  } else if (ha && hb) {
    TRACE_BGEMM(false, false, true, true);
  } else if (ha) {
    TRACE_BGEMM(false, false, true, false);
  } else if (hb) {
    TRACE_BGEMM(false, false, false, true);
  } else {
    TRACE_BGEMM(false, false, false, false);
  }
#undef TRACE_BGEMM
}

}  // namespace

int64_t bgemm_ws_floats(int M, int N, int K) {
  const int s = std::max(bgemm_splits(M, N, (int)rup(K, BK)), big::splits(M, N, (int)rup(K, big::TK)));
  return s > 1 ? (int64_t)s * M * N : 0;
}

bool launch_bgemm(const GemmArgs& g, const GemmArgs* g2, float* ws, int64_t ws_cap, hipStream_t s, int force) {
  if (!g.roundA && !g.roundB) return false;  // fp32 operands on both sides: not this kernel
  if (g2 && (g2->M != g.M || g2->N != g.N || g2->roundA != g.roundA || g2->roundB != g.roundB ||
             g2->halfA != g.halfA || g2->halfB != g.halfB))
    return false;
  // a bf16-stored operand is a storage point (rounded), never split
  if ((g.halfA && !g.roundA) || (g.halfB && !g.roundB)) return false;
  Src A{}, B{};
  bool akc = false, bkc = false;
  if (!add_segment(A, 0, g.A, g.sam, g.sak, g.M, g.K, akc, g.halfA)) return false;
  if (!add_segment(B, 0, g.B, g.sbn, g.sbk, g.N, g.K, bkc, g.halfB)) return false;
  if (g2) {
    if (!add_segment(A, 1, g2->A, g2->sam, g2->sak, g.M, g2->K, akc, g.halfA)) return false;
    if (!add_segment(B, 1, g2->B, g2->sbn, g2->sbk, g.N, g2->K, bkc, g.halfB)) return false;
  } else {
    A.p1 = A.p0;
    A.ld1 = A.ld0;
    B.p1 = B.p0;
    B.ld1 = B.ld0;
  }
  if (g.r1c) {  // rank-one rows: B fp32 with its rows contiguous, split, one segment
    if (g2 || bkc || g.halfB || g.roundB || g.sbn != 1 || g.N % 4 != 0 || g.r1dsh < 2 || g.r1H <= 0) return false;
    B.r1c = g.r1c;
    B.r1tsh = g.r1tsh;
    B.r1dsh = g.r1dsh;
    B.r1H = g.r1H;
    B.r1round = g.r1round;
    B.r1scale = g.r1scale;
  }
  const int K0 = g.K, K1 = g2 ? g2->K : 0;
  if (K0 + K1 == 0) return false;
  if (g.gelu_u && (g.beta != 0.f || g2)) return false;
  if (g.halfC && (g.beta != 0.f || (g.ldc & 3) != 0)) return false;
  const bool sa = !g.roundA, sb = !g.roundB, ha = g.halfA != 0, hb = g.halfB != 0;
  // the 256-tile kernel when it fills the chip, else the 128-tile one; stages
  // are aligned to each kernel's k step, and so is the start of segment 1
  const int kpb = (int)(rup(K0, big::TK) + rup(K1, big::TK));
  int splits = big::splits(g.M, g.N, kpb);
  bool use_big = splits > 0;
  if (force == 1) use_big = false;
  if (force == 2 && !use_big) {
    use_big = true;
    splits = 1;
  }
  const int step = use_big ? big::TK : BK;
  A.k1p = B.k1p = (int)rup(K0, step);
  const int Kp = (int)(rup(K0, step) + rup(K1, step));
  if (!use_big) splits = bgemm_splits(g.M, g.N, Kp);
  while (splits > 1 && (int64_t)splits * g.M * g.N > ws_cap) splits /= 2;
  if (g.gelu_u || g.halfC) splits = 1;  // the epilogue needs the whole sum
  const int kchunk = (int)rup((Kp + splits - 1) / splits, step);
  splits = (Kp + kchunk - 1) / kchunk;
  float* part = splits > 1 ? ws : nullptr;
  const int TMk = use_big ? big::TM : BM, TNk = use_big ? big::TN : BN;
  const int tn = (int)(rup(g.N, TNk) / TNk), tm = (int)(rup(g.M, TMk) / TMk);
  const dim3 grid((unsigned)(tn * tm * splits));
  if (use_big) {
    if (akc && bkc)
      big::launch_orient<true, true>(sa, sb, ha, hb, grid, A, B, Kp, g, part, kchunk, tn, tm, s);
    else if (akc)
      big::launch_orient<true, false>(sa, sb, ha, hb, grid, A, B, Kp, g, part, kchunk, tn, tm, s);
    else if (bkc)
      big::launch_orient<false, true>(sa, sb, ha, hb, grid, A, B, Kp, g, part, kchunk, tn, tm, s);
    else
      big::launch_orient<false, false>(sa, sb, ha, hb, grid, A, B, Kp, g, part, kchunk, tn, tm, s);
  } else {
    if (akc && bkc)
      launch_orient<true, true>(sa, sb, ha, hb, grid, A, B, Kp, g, part, kchunk, tn, tm, s);
    else if (akc)
      launch_orient<true, false>(sa, sb, ha, hb, grid, A, B, Kp, g, part, kchunk, tn, tm, s);
    else if (bkc)
      launch_orient<false, true>(sa, sb, ha, hb, grid, A, B, Kp, g, part, kchunk, tn, tm, s);
    else
      launch_orient<false, false>(sa, sb, ha, hb, grid, A, B, Kp, g, part, kchunk, tn, tm, s);
  }
  if (splits > 1) launch_splitk_reduce(ws, splits, g.M, g.N, g.C, g.ldc, g.beta, g.Cin, s);
  return true;
}
