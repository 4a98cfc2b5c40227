// GEMM of the update step on bf16 operands (Alg. 1: the backward of the
// estimator's loss, every product of which is a plain matrix product).
//
// Each operand is first written by a memory-bound prep kernel as a bf16 copy
// whose contiguous dimension is k (rows = m for A, n for B), zero-padded to
// whole tiles; operands that are fp32 values rather than bf16 storage points
// are split into hi = bf16(v) and lo = bf16(v - hi), and their products take
// two MFMAs (hi.B + lo.B), which keeps about 16 significant bits of v.
// The GEMM then moves 128 x 64 operand tiles straight from global memory to
// LDS (16-byte direct loads, no register staging), double-buffered, in an
// XOR-swizzled layout that makes the 16-byte fragment reads conflict-free,
// and runs 16x16x32 bf16 MFMAs on 64x64 blocks per wave.  Split-K partial
// sums go to a workspace and are added in a fixed order, so results do not
// depend on scheduling.
#include "kcommon.h"
#include "kernels.h"

namespace {

constexpr int BM = 128, BN = 128, BK = 64;
constexpr int UNITS = BM * BK * 2 / 16;  // 16-byte units per 128 x 64 bf16 tile (1024)

inline int64_t rup(int64_t x, int64_t a) { return (x + a - 1) / a * a; }

__device__ __forceinline__ void split_bf(float v, uint16_t& h, uint16_t& l) {
  h = f2bf(v);
  l = f2bf(v - bf2f(h));
}

// out[c][r] = bf16(src[r*ld + c]) for r < R, c < C, zero elsewhere: rows
// [0, rows_p) of length Kp (k = r).  64 x 64 source tiles through LDS, so that
// both the reads (along c) and the writes (along r) are coalesced.
__global__ __launch_bounds__(256) void k_prep_t(const float* __restrict__ src, int R, int C, int64_t ld,
                                                uint16_t* __restrict__ hi, uint16_t* __restrict__ lo, int Kp) {
  __shared__ float t[64][65];
  const int r0 = blockIdx.x * 64, c0 = blockIdx.y * 64, tid = threadIdx.x;
#pragma unroll
  for (int q = 0; q < 16; ++q) {
    const int idx = tid + q * 256, rr = idx >> 6, cc = idx & 63;
    const int r = r0 + rr, c = c0 + cc;
    t[rr][cc] = (r < R && c < C) ? src[(int64_t)r * ld + c] : 0.f;
  }
  __syncthreads();
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    const int u = tid + q * 256, i = u >> 3, kc = u & 7;
    uint16_t h[8], l[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) split_bf(t[kc * 8 + j][i], h[j], l[j]);
    const int64_t o = (int64_t)(c0 + i) * Kp + r0 + kc * 8;
    *reinterpret_cast<uint4*>(hi + o) = make_uint4(h[0] | (uint32_t)h[1] << 16, h[2] | (uint32_t)h[3] << 16,
                                                   h[4] | (uint32_t)h[5] << 16, h[6] | (uint32_t)h[7] << 16);
    if (lo)
      *reinterpret_cast<uint4*>(lo + o) = make_uint4(l[0] | (uint32_t)l[1] << 16, l[2] | (uint32_t)l[3] << 16,
                                                     l[4] | (uint32_t)l[5] << 16, l[6] | (uint32_t)l[7] << 16);
  }
}

// out[r][c] = bf16(src[r*ld + c]) for r < R, c < C, zero elsewhere: rows
// [0, rows_p) of length Kp (k = c); eight elements per thread.
__global__ __launch_bounds__(256) void k_prep_n(const float* __restrict__ src, int R, int C, int64_t ld,
                                                uint16_t* __restrict__ hi, uint16_t* __restrict__ lo, int rows_p,
                                                int Kp) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int kcn = Kp / 8;
  if (i >= (int64_t)rows_p * kcn) return;
  const int r = (int)(i / kcn), c0 = (int)(i % kcn) * 8;
  uint16_t h[8], l[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) split_bf((r < R && c0 + j < C) ? src[(int64_t)r * ld + c0 + j] : 0.f, h[j], l[j]);
  const int64_t o = (int64_t)r * Kp + c0;
  *reinterpret_cast<uint4*>(hi + o) = make_uint4(h[0] | (uint32_t)h[1] << 16, h[2] | (uint32_t)h[3] << 16,
                                                 h[4] | (uint32_t)h[5] << 16, h[6] | (uint32_t)h[7] << 16);
  if (lo)
    *reinterpret_cast<uint4*>(lo + o) = make_uint4(l[0] | (uint32_t)l[1] << 16, l[2] | (uint32_t)l[3] << 16,
                                                   l[4] | (uint32_t)l[5] << 16, l[6] | (uint32_t)l[7] << 16);
}

// LDS unit (16 bytes) of (row, k-chunk c) in a swizzled 128 x 64 tile.
__device__ __forceinline__ int unit_of(int row, int c) { return row * 8 + (c ^ (row & 7)); }

// 128 x 64 tile of a prepared operand (rows row0.., k k0..) -> LDS tile, by
// 16 direct 1 KiB loads; this wave issues loads q = wave*4 .. wave*4 + 3.
__device__ __forceinline__ void tile_to_lds(const uint16_t* __restrict__ op, int64_t Kp, int row0, int k0,
                                            uint4* dst, int wave, int lane) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int q = wave * 4 + i;
    const int u = q * 64 + lane, row = u >> 3, c = (u & 7) ^ (row & 7);
    __builtin_amdgcn_global_load_lds((const void*)(op + (int64_t)(row0 + row) * Kp + k0 + c * 8),
                                     (__attribute__((address_space(3))) void*)(dst + q * 64), 16, 0, 0);
  }
}

// C[m][n] (+)= sum_k A[m][k] B[n][k] over this split's k range, operands
// prepared (bf16, k contiguous, padded); SA / SB: that operand has a lo part.
template <bool SA, bool SB>
__global__ __launch_bounds__(256) void k_bgemm(const uint16_t* __restrict__ Ah, const uint16_t* __restrict__ Al,
                                               const uint16_t* __restrict__ Bh, const uint16_t* __restrict__ Bl,
                                               int Kp, int M, int N, float* C, int64_t ldc, float beta,
                                               float* __restrict__ part, int kchunk) {
  static_assert(!(SA && SB), "at most one operand is split");
  constexpr int NT = 2 + (SA ? 1 : 0) + (SB ? 1 : 0);  // tiles per stage: A hi, B hi, [A lo | B lo]
  __shared__ uint4 lds[2][NT][UNITS];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, lg = lane >> 4, lc = lane & 15;
  const int wm = wave >> 1, wn = wave & 1;
  const int m0 = blockIdx.y * BM, n0 = blockIdx.x * BN;
  const int kb = blockIdx.z * kchunk;
  const int ke = min(Kp, kb + kchunk);
  f32x4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  auto stage = [&](int buf, int k0) {
    tile_to_lds(Ah, Kp, m0, k0, lds[buf][0], wave, lane);
    tile_to_lds(Bh, Kp, n0, k0, lds[buf][1], wave, lane);
    if constexpr (SA) tile_to_lds(Al, Kp, m0, k0, lds[buf][2], wave, lane);
    if constexpr (SB) tile_to_lds(Bl, Kp, n0, k0, lds[buf][NT - 1], wave, lane);
  };
  if (kb < ke) stage(0, kb);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  int buf = 0;
  for (int k0 = kb; k0 < ke; k0 += BK, buf ^= 1) {
    if (k0 + BK < ke) stage(buf ^ 1, k0 + BK);
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
    __builtin_amdgcn_s_waitcnt(0);  // this wave's part of the next stage has landed
    __syncthreads();
  }
  // lane holds C[m0 + wm*64 + rf*16 + 4*lg + r][n0 + wn*64 + nf*16 + lc]
#pragma unroll
  for (int rf = 0; rf < 4; ++rf)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int m = m0 + wm * 64 + rf * 16 + 4 * lg + r;
      if (m >= M) continue;
#pragma unroll
      for (int nf = 0; nf < 4; ++nf) {
        const int n = n0 + wn * 64 + nf * 16 + lc;
        if (n >= N) continue;
        if (part) {
          part[((int64_t)blockIdx.z * M + m) * N + n] = acc[rf][nf][r];
        } else {
          float* cp = C + (int64_t)m * ldc + n;
          *cp = (beta != 0.f) ? (*cp + acc[rf][nf][r]) : acc[rf][nf][r];
        }
      }
    }
}

// One operand (rows x K, element (row, k) at src[row*srow + k*sk], one of the
// strides 1) -> prepared copy at hi (and lo when split).
void prep(const float* src, int rows, int K, int64_t srow, int64_t sk, bool split, uint16_t* hi, uint16_t* lo,
          hipStream_t s) {
  const int rows_p = (int)rup(rows, 128), Kp = (int)rup(K, BK);
  if (sk == 1) {
    const int64_t n = (int64_t)rows_p * (Kp / 8);
    hipLaunchKernelGGL(k_prep_n, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, src, rows, K, srow, hi,
                       split ? lo : nullptr, rows_p, Kp);
  } else {
    // src is [K][rows] with row stride sk: transpose into [rows][K]
    hipLaunchKernelGGL(k_prep_t, dim3((unsigned)(Kp / 64), (unsigned)(rows_p / 64)), dim3(256), 0, s, src, K, rows,
                       sk, hi, split ? lo : nullptr, Kp);
  }
}

int bgemm_splits(int M, int N, int Kp) {
  const int tiles = (int)(rup(M, BM) / BM * (rup(N, BN) / BN));
  int splits = 1;
  // fill the 256 CUs about twice, each split keeping at least 512 k values
  // (shorter splits measured slower: the partial sums cost more than they fill)
  while (tiles * splits < 512 && Kp / (splits * 2) >= 512) splits *= 2;
  return splits;
}

}  // namespace

int64_t bgemm_prep_bytes(int M, int N, int K) {
  const int64_t Kp = rup(K, BK);
  return 2 * (rup(M, BM) * Kp * 2) + 2 * (rup(N, BN) * Kp * 2) + 256;
}
int64_t bgemm_ws_floats(int M, int N, int K) {
  const int s = bgemm_splits(M, N, (int)rup(K, BK));
  return s > 1 ? (int64_t)s * M * N : 0;
}

bool launch_bgemm(const GemmArgs& g, float* ws, int64_t ws_cap, void* prep_buf, int64_t prep_cap, hipStream_t s) {
  if (!g.roundA && !g.roundB) return false;  // fp32 operands on both sides: not this kernel
  if (!((g.sak == 1 || g.sam == 1) && (g.sbk == 1 || g.sbn == 1))) return false;
  if (!prep_buf || bgemm_prep_bytes(g.M, g.N, g.K) > prep_cap) return false;
  const bool sa = !g.roundA, sb = !g.roundB;
  const int Kp = (int)rup(g.K, BK);
  const int64_t asz = rup(g.M, BM) * Kp, bsz = rup(g.N, BN) * Kp;  // elements per part
  uint16_t* p = (uint16_t*)prep_buf;
  uint16_t *Ah = p, *Al = p + asz, *Bh = p + 2 * asz, *Bl = p + 2 * asz + bsz;
  // A(m, k) = A[m*sam + k*sak]; B(k, n) = B[k*sbk + n*sbn] is row n of B^T
  prep(g.A, g.M, g.K, g.sak == 1 ? g.sam : 1, g.sak == 1 ? 1 : g.sak, sa, Ah, Al, s);
  prep(g.B, g.N, g.K, g.sbk == 1 ? g.sbn : 1, g.sbk == 1 ? 1 : g.sbk, sb, Bh, Bl, s);
  int splits = bgemm_splits(g.M, g.N, Kp);
  while (splits > 1 && (int64_t)splits * g.M * g.N > ws_cap) splits /= 2;
  const int kchunk = (int)rup((Kp + splits - 1) / splits, BK);
  float* part = splits > 1 ? ws : nullptr;
  const dim3 grid((unsigned)(rup(g.N, BN) / BN), (unsigned)(rup(g.M, BM) / BM), (unsigned)splits);
  if (sa)
    hipLaunchKernelGGL((k_bgemm<true, false>), grid, dim3(256), 0, s, Ah, Al, Bh, Bl, Kp, g.M, g.N, g.C, g.ldc,
                       g.beta, part, kchunk);
  else if (sb)
    hipLaunchKernelGGL((k_bgemm<false, true>), grid, dim3(256), 0, s, Ah, Al, Bh, Bl, Kp, g.M, g.N, g.C, g.ldc,
                       g.beta, part, kchunk);
  else
    hipLaunchKernelGGL((k_bgemm<false, false>), grid, dim3(256), 0, s, Ah, Al, Bh, Bl, Kp, g.M, g.N, g.C, g.ldc,
                       g.beta, part, kchunk);
  if (splits > 1) launch_splitk_reduce(ws, splits, g.M, g.N, g.C, g.ldc, g.beta, s);
  return true;
}
