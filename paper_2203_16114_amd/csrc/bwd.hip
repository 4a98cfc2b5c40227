// Gated adaptation on gfx950: the gradient of the batch-mean cross-entropy
// through the forward of fwd.hip (Model.backward of Alg. 1, line 10), and the
// Adam update (Sec. 6: Adam, lr 0.001).  Every reduction runs in a fixed order,
// so two runs on the same inputs give bitwise-identical gradients: split-K
// partial products, column sums and embedding-gradient partial tables are
// combined by a second pass that adds them in index order.
#include "kcommon.h"
#include "kernels.h"

#include <hip/hip_ext.h>

// ------------------------------------------------------------ generic GEMM ----
// C(m,n) [+]= sum_k A(m,k) B(k,n) for arbitrary element strides.  64x64 output
// tile per workgroup, 4 waves in a 2x2 layout of 32x32 sub-tiles; the k range
// is walked in steps of 32 staged through LDS as [row][k] (A) and [col][k] (B)
// so that both fragments are 16-byte LDS reads.  Operands are rounded to bf16
// on the way into LDS where the caller asks (the bf16 storage points).
template <bool BF>
__global__ __launch_bounds__(256) void k_gemm(GemmArgs g, float* __restrict__ part, int kchunk) {
  typedef Mma<BF> M;
  typedef typename M::T OT;
  constexpr int BM = 64, BN = 64, BK = 32;
  constexpr int STR = BK * (int)sizeof(OT) + 16;
  __shared__ __align__(16) unsigned char As[BM * STR];
  __shared__ __align__(16) unsigned char Bs[BN * STR];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, lg = lane >> 4, lc = lane & 15;
  const int wm = wave >> 1, wn = wave & 1;
  const int m0 = blockIdx.y * BM, n0 = blockIdx.x * BN;
  const int kbeg = blockIdx.z * kchunk;
  const int kend = min(g.K, kbeg + kchunk);
  f32x4 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  const bool a_k_fast = (g.sak == 1);
  const bool b_n_fast = (g.sbn == 1);
  for (int k0 = kbeg; k0 < kend; k0 += BK) {
#pragma unroll
    for (int it = 0; it < (BM * BK) / 256; ++it) {
      const int i = tid + it * 256;
      int mm, kk;
      if (a_k_fast) {
        mm = i / BK;
        kk = i % BK;
      } else {
        kk = i / BM;
        mm = i % BM;
      }
      const int m = m0 + mm, k = k0 + kk;
      float v = (m < g.M && k < kend) ? g.A[(int64_t)m * g.sam + (int64_t)k * g.sak] : 0.f;
      if (g.roundA) v = round_bf(v);
      ((OT*)(As + mm * STR))[kk] = M::cvt(v);
    }
#pragma unroll
    for (int it = 0; it < (BN * BK) / 256; ++it) {
      const int i = tid + it * 256;
      int nn, kk;
      if (b_n_fast) {
        kk = i / BN;
        nn = i % BN;
      } else {
        nn = i / BK;
        kk = i % BK;
      }
      const int n = n0 + nn, k = k0 + kk;
      float v = (n < g.N && k < kend) ? g.B[(int64_t)k * g.sbk + (int64_t)n * g.sbn] : 0.f;
      if (g.roundB) v = round_bf(v);
      ((OT*)(Bs + nn * STR))[kk] = M::cvt(v);
    }
    __syncthreads();
#pragma unroll
    for (int ks = 0; ks < BK / M::KS; ++ks) {
      uint4 af[2], bfr[2];
#pragma unroll
      for (int rf = 0; rf < 2; ++rf) af[rf] = *(const uint4*)(As + (wm * 32 + rf * 16 + lc) * STR + ks * 64 + lg * 16);
#pragma unroll
      for (int nf = 0; nf < 2; ++nf) bfr[nf] = *(const uint4*)(Bs + (wn * 32 + nf * 16 + lc) * STR + ks * 64 + lg * 16);
#pragma unroll
      for (int rf = 0; rf < 2; ++rf)
#pragma unroll
        for (int nf = 0; nf < 2; ++nf) M::run(acc[rf][nf], af[rf], bfr[nf]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int rf = 0; rf < 2; ++rf)
#pragma unroll
    for (int nf = 0; nf < 2; ++nf)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = m0 + wm * 32 + rf * 16 + 4 * lg + r;
        const int n = n0 + wn * 32 + nf * 16 + lc;
        if (m < g.M && n < g.N) {
          if (part) {
            part[((int64_t)blockIdx.z * g.M + m) * g.N + n] = acc[rf][nf][r];
          } else {
            float* c = g.C + (int64_t)m * g.ldc + n;
            *c = (g.beta != 0.f) ? (*c + acc[rf][nf][r]) : acc[rf][nf][r];
          }
        }
      }
}

// C(m,n) = [C(m,n) +] sum_z part[z][m][n], z in increasing order.
__global__ void k_splitk_reduce(const float* __restrict__ part, int splits, int M, int N, float* C, int64_t ldc,
                                float beta, const float* cin) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= (int64_t)M * N) return;
  const int m = (int)(i / N), n = (int)(i % N);
  float s = 0.f;
  for (int z = 0; z < splits; ++z) s += part[((int64_t)z * M + m) * N + n];
  const int64_t o = (int64_t)m * ldc + n;
  C[o] = (beta != 0.f) ? (cin[o] + s) : s;
}

// 128x128-tile GEMM for the two operand layouts of the update: operands whose
// contiguous dimension is k (activation gradients, dY . W^T) and operands
// whose contiguous dimension is m or n (weight gradients, act^T . dY).  Global
// reads are float4 along the contiguous dimension; the next k-tile is held in
// registers while the current one is multiplied from LDS (two LDS buffers,
// one barrier per k-tile).  Modes:
//   GM_F32      both operands fp32 (fp32 models): 16x16x4 fp32 MFMA;
//   GM_BF16     both operands at a bf16 storage point: 16x16x32 bf16 MFMA;
//   GM_SPLIT_A  A is an fp32 value, B a bf16 storage point: A = hi + lo with
//   GM_SPLIT_B  hi = bf16(A), lo = bf16(A - hi), two bf16 MFMAs per product
//               (the fp32 operand keeps ~16 significant bits; 2^-17 relative).
enum { GM_F32 = 0, GM_BF16 = 1, GM_SPLIT_A = 2, GM_SPLIT_B = 3 };

template <int MODE>
__device__ __forceinline__ void st_lds(unsigned char* row_hi, unsigned char* row_lo, int k, float v, bool split,
                                       bool rnd) {
  if constexpr (MODE == GM_F32) {
    ((float*)row_hi)[k] = v;
  } else {
    const uint16_t h = f2bf(v);
    ((uint16_t*)row_hi)[k] = h;
    if (split) ((uint16_t*)row_lo)[k] = f2bf(v - bf2f(h));
    (void)rnd;
  }
}

template <int MODE, bool AK, bool BKF>
__global__ __launch_bounds__(256) void k_gemm128(GemmArgs g, float* __restrict__ part, int kchunk) {
  constexpr bool BFOP = MODE != GM_F32;
  typedef Mma<BFOP> M;
  typedef typename M::T OT;
  constexpr int BM = 128, BN = 128, BK = 32;
  constexpr int STR = BK * (int)sizeof(OT) + 16;
  constexpr bool SPA = MODE == GM_SPLIT_A, SPB = MODE == GM_SPLIT_B;
  constexpr int AT = BM * STR, BT = BN * STR;
  __shared__ __align__(16) unsigned char As[2][(SPA ? 2 : 1) * AT];
  __shared__ __align__(16) unsigned char Bs[2][(SPB ? 2 : 1) * BT];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, lg = lane >> 4, lc = lane & 15;
  const int wm = wave >> 1, wn = wave & 1;
  const int m0 = blockIdx.y * BM, n0 = blockIdx.x * BN;
  const int kbeg = blockIdx.z * kchunk;
  const int kend = min(g.K, kbeg + kchunk);
  f32x4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  float4 ra[4], rb[4];
  // element (row, k) of the tile loaded by float4 q: see the index maps below
  auto load = [&](int k0) {
#pragma unroll
    for (int it = 0; it < 4; ++it) {
      const int q = tid + it * 256;
      if (AK) {
        const int mm = q >> 3, kk = (q & 7) * 4;
        const int m = m0 + mm, k = k0 + kk;
        if (m < g.M && k + 3 < kend) {
          ra[it] = *reinterpret_cast<const float4*>(g.A + (int64_t)m * g.sam + k);
        } else {
          float t[4];
#pragma unroll
          for (int u = 0; u < 4; ++u) t[u] = (m < g.M && k + u < kend) ? g.A[(int64_t)m * g.sam + k + u] : 0.f;
          ra[it] = make_float4(t[0], t[1], t[2], t[3]);
        }
      } else {
        const int kk = q >> 5, mm = (q & 31) * 4;
        const int m = m0 + mm, k = k0 + kk;
        ra[it] = (k < kend && m < g.M) ? *reinterpret_cast<const float4*>(g.A + m + (int64_t)k * g.sak)
                                       : make_float4(0.f, 0.f, 0.f, 0.f);
      }
      if (BKF) {
        const int nn = q >> 3, kk = (q & 7) * 4;
        const int n = n0 + nn, k = k0 + kk;
        if (n < g.N && k + 3 < kend) {
          rb[it] = *reinterpret_cast<const float4*>(g.B + k + (int64_t)n * g.sbn);
        } else {
          float t[4];
#pragma unroll
          for (int u = 0; u < 4; ++u) t[u] = (n < g.N && k + u < kend) ? g.B[k + u + (int64_t)n * g.sbn] : 0.f;
          rb[it] = make_float4(t[0], t[1], t[2], t[3]);
        }
      } else {
        const int kk = q >> 5, nn = (q & 31) * 4;
        const int n = n0 + nn, k = k0 + kk;
        rb[it] = (k < kend && n < g.N) ? *reinterpret_cast<const float4*>(g.B + (int64_t)k * g.sbk + n)
                                       : make_float4(0.f, 0.f, 0.f, 0.f);
      }
    }
  };
  auto store = [&](int buf) {
    unsigned char* Ah = As[buf];
    unsigned char* Al = As[buf] + (SPA ? AT : 0);
    unsigned char* Bh = Bs[buf];
    unsigned char* Bl = Bs[buf] + (SPB ? BT : 0);
#pragma unroll
    for (int it = 0; it < 4; ++it) {
      const int q = tid + it * 256;
      const float va[4] = {ra[it].x, ra[it].y, ra[it].z, ra[it].w};
      const float vb[4] = {rb[it].x, rb[it].y, rb[it].z, rb[it].w};
      if (AK) {
        const int mm = q >> 3, kk = (q & 7) * 4;
#pragma unroll
        for (int u = 0; u < 4; ++u) st_lds<MODE>(Ah + mm * STR, Al + mm * STR, kk + u, va[u], SPA, true);
      } else {
        const int kk = q >> 5, mm = (q & 31) * 4;
#pragma unroll
        for (int u = 0; u < 4; ++u) st_lds<MODE>(Ah + (mm + u) * STR, Al + (mm + u) * STR, kk, va[u], SPA, true);
      }
      if (BKF) {
        const int nn = q >> 3, kk = (q & 7) * 4;
#pragma unroll
        for (int u = 0; u < 4; ++u) st_lds<MODE>(Bh + nn * STR, Bl + nn * STR, kk + u, vb[u], SPB, true);
      } else {
        const int kk = q >> 5, nn = (q & 31) * 4;
#pragma unroll
        for (int u = 0; u < 4; ++u) st_lds<MODE>(Bh + (nn + u) * STR, Bl + (nn + u) * STR, kk, vb[u], SPB, true);
      }
    }
  };
  if (kbeg < kend) {
    load(kbeg);
    store(0);
  }
  __syncthreads();
  int it = 0;
  for (int k0 = kbeg; k0 < kend; k0 += BK, ++it) {
    const int cur = it & 1;
    const bool more = k0 + BK < kend;
    if (more) load(k0 + BK);
    const unsigned char* Ah = As[cur];
    const unsigned char* Bh = Bs[cur];
#pragma unroll
    for (int ks = 0; ks < BK / M::KS; ++ks) {
      uint4 af[4], bfr[4];
#pragma unroll
      for (int rf = 0; rf < 4; ++rf) af[rf] = *(const uint4*)(Ah + (wm * 64 + rf * 16 + lc) * STR + ks * 64 + lg * 16);
#pragma unroll
      for (int nf = 0; nf < 4; ++nf) bfr[nf] = *(const uint4*)(Bh + (wn * 64 + nf * 16 + lc) * STR + ks * 64 + lg * 16);
#pragma unroll
      for (int rf = 0; rf < 4; ++rf)
#pragma unroll
        for (int nf = 0; nf < 4; ++nf) M::run(acc[rf][nf], af[rf], bfr[nf]);
      if constexpr (SPA) {
#pragma unroll
        for (int rf = 0; rf < 4; ++rf)
          af[rf] = *(const uint4*)(Ah + AT + (wm * 64 + rf * 16 + lc) * STR + ks * 64 + lg * 16);
#pragma unroll
        for (int rf = 0; rf < 4; ++rf)
#pragma unroll
          for (int nf = 0; nf < 4; ++nf) M::run(acc[rf][nf], af[rf], bfr[nf]);
      }
      if constexpr (SPB) {
#pragma unroll
        for (int nf = 0; nf < 4; ++nf)
          bfr[nf] = *(const uint4*)(Bh + BT + (wn * 64 + nf * 16 + lc) * STR + ks * 64 + lg * 16);
#pragma unroll
        for (int rf = 0; rf < 4; ++rf)
#pragma unroll
          for (int nf = 0; nf < 4; ++nf) M::run(acc[rf][nf], af[rf], bfr[nf]);
      }
    }
    if (more) store(cur ^ 1);
    __syncthreads();
  }
#pragma unroll
  for (int rf = 0; rf < 4; ++rf)
#pragma unroll
    for (int nf = 0; nf < 4; ++nf)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = m0 + wm * 64 + rf * 16 + 4 * lg + r;
        const int n = n0 + wn * 64 + nf * 16 + lc;
        if (m < g.M && n < g.N) {
          if (part) {
            part[((int64_t)blockIdx.z * g.M + m) * g.N + n] = acc[rf][nf][r];
          } else {
            float* c = g.C + (int64_t)m * g.ldc + n;
            *c = (g.beta != 0.f) ? (*c + acc[rf][nf][r]) : acc[rf][nf][r];
          }
        }
      }
}

static int gemm_splits(int M, int N, int K) {
  const int tiles = ((M + 127) / 128) * ((N + 127) / 128);
  int splits = 1;
  // enough workgroups to fill 256 CUs twice, each split still covering >= 256 k values
  while (tiles * splits < 512 && (K + splits * 2 - 1) / (splits * 2) >= 256) splits *= 2;
  return splits;
}
int64_t gemm_ws_floats(int M, int N, int K) {
  const int s = gemm_splits(M, N, K);
  return s > 1 ? (int64_t)s * M * N : 0;
}
static bool aligned16(const void* p) { return ((uintptr_t)p & 15) == 0; }

template <int MODE>
static void launch128(const GemmArgs& g, float* part, int kchunk, dim3 grid, hipStream_t s) {
  const bool ak = g.sak == 1, bk = g.sbk == 1;
  if (ak && bk)
    hipLaunchKernelGGL((k_gemm128<MODE, true, true>), grid, dim3(256), 0, s, g, part, kchunk);
  else if (ak)
    hipLaunchKernelGGL((k_gemm128<MODE, true, false>), grid, dim3(256), 0, s, g, part, kchunk);
  else if (bk)
    hipLaunchKernelGGL((k_gemm128<MODE, false, true>), grid, dim3(256), 0, s, g, part, kchunk);
  else
    hipLaunchKernelGGL((k_gemm128<MODE, false, false>), grid, dim3(256), 0, s, g, part, kchunk);
}

// Four consecutive n per thread (one float4 of C and of each partial), eight
// partials in flight; the same sum order (z increasing, then the addend) as
// k_splitk_reduce.  Needs N, ldc multiples of 4 and 16-byte aligned C, cin.
__global__ __launch_bounds__(256) void k_splitk_reduce4(const float* __restrict__ part, int splits, int M, int N,
                                                        float* C, int64_t ldc, float beta, const float* cin) {
  const uint32_t q = blockIdx.x * 256u + threadIdx.x, n4 = (uint32_t)N >> 2;
  if (q >= (uint32_t)M * n4) return;
  const uint32_t m = q / n4, n = (q - m * n4) * 4;
  const int64_t MN = (int64_t)M * N;
  const float* p = part + (int64_t)m * N + n;
  float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
  auto add = [&](const float4& v) {
    s.x += v.x;
    s.y += v.y;
    s.z += v.z;
    s.w += v.w;
  };
  int z = 0;
  for (; z + 8 <= splits; z += 8) {
    float4 v[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) v[j] = *reinterpret_cast<const float4*>(p + (int64_t)(z + j) * MN);
#pragma unroll
    for (int j = 0; j < 8; ++j) add(v[j]);
  }
  for (; z < splits; ++z) add(*reinterpret_cast<const float4*>(p + (int64_t)z * MN));
  const int64_t o = (int64_t)m * ldc + n;
  if (beta != 0.f) add(*reinterpret_cast<const float4*>(cin + o));
  *reinterpret_cast<float4*>(C + o) = s;
}

void launch_splitk_reduce(const float* ws, int splits, int M, int N, float* C, int64_t ldc, float beta,
                          const float* cin, hipStream_t s) {
  if (!cin) cin = C;
  const int64_t tot = (int64_t)M * N;
  if (N % 4 == 0 && ldc % 4 == 0 && ((uintptr_t)ws & 15) == 0 && ((uintptr_t)C & 15) == 0 &&
      ((uintptr_t)cin & 15) == 0)
    hipLaunchKernelGGL(k_splitk_reduce4, dim3((unsigned)((tot / 4 + 255) / 256)), dim3(256), 0, s, ws, splits, M, N, C,
                       ldc, beta, cin);
  else
    hipLaunchKernelGGL(k_splitk_reduce, dim3((unsigned)((tot + 255) / 256)), dim3(256), 0, s, ws, splits, M, N, C, ldc,
                       beta, cin);
}

bool launch_gemm(const GemmArgs& g0, float* ws, int64_t ws_cap, hipStream_t s) {
  if (g0.M <= 0 || g0.N <= 0) return true;
  // bf16 storage points on at least one side: register-staged bf16 GEMM
  if (launch_bgemm(g0, nullptr, ws, ws_cap, s)) return true;
  // the kernels below use fp32 operands and results, and read B as stored
  if (g0.halfA || g0.halfB || g0.halfC || g0.r1c) return false;
  GemmArgs g = g0;
  if (g.Cin && g.Cin != g.C && g.beta != 0.f) {  // the kernels below add C itself: the addend goes there first
    (void)hipMemcpy2DAsync(g.C, (size_t)g.ldc * 4, g.Cin, (size_t)g.ldc * 4, (size_t)g.N * 4, (size_t)g.M,
                           hipMemcpyDeviceToDevice, s);
  }
  g.Cin = nullptr;
  if (g.gelu_u) {  // the product, then the GELU derivative in place (C laid out densely, as gelu_u)
    GemmArgs h = g;
    h.gelu_u = nullptr;
    launch_gemm(h, ws, ws_cap, s);
    launch_gelu_bwd(g.C, g.gelu_u, g.C, (int64_t)g.M * g.N, s);
    return true;
  }
  int splits = gemm_splits(g.M, g.N, g.K);
  while (splits > 1 && (int64_t)splits * g.M * g.N > ws_cap) splits /= 2;
  int kchunk = (g.K + splits - 1) / splits;
  kchunk = (kchunk + 31) / 32 * 32;
  float* part = splits > 1 ? ws : nullptr;
  // the 128-tile kernel needs float4 access along each operand's contiguous dimension
  const bool a_ok = aligned16(g.A) && ((g.sak == 1 && g.sam % 4 == 0) || (g.sam == 1 && g.sak % 4 == 0 && g.M % 4 == 0));
  const bool b_ok = aligned16(g.B) && ((g.sbk == 1 && g.sbn % 4 == 0) || (g.sbn == 1 && g.sbk % 4 == 0 && g.N % 4 == 0));
  if (a_ok && b_ok) {
    const dim3 grid((g.N + 127) / 128, (g.M + 127) / 128, splits);
    if (g.roundA && g.roundB)
      launch128<GM_BF16>(g, part, kchunk, grid, s);
    else if (!g.roundA && !g.roundB)
      launch128<GM_F32>(g, part, kchunk, grid, s);
    else if (g.roundB)
      launch128<GM_SPLIT_A>(g, part, kchunk, grid, s);
    else
      launch128<GM_SPLIT_B>(g, part, kchunk, grid, s);
  } else {
    const dim3 grid((g.N + 63) / 64, (g.M + 63) / 64, splits);
    if (g.roundA && g.roundB)
      hipLaunchKernelGGL(k_gemm<true>, grid, dim3(256), 0, s, g, part, kchunk);
    else
      hipLaunchKernelGGL(k_gemm<false>, grid, dim3(256), 0, s, g, part, kchunk);
  }
  if (splits > 1) launch_splitk_reduce(ws, splits, g.M, g.N, g.C, g.ldc, g.beta, nullptr, s);
  return true;
}

void launch_gemm2(const GemmArgs& g, const GemmArgs& g2, float* ws, int64_t ws_cap, hipStream_t s) {
  if (g.M <= 0 || g.N <= 0) return;
  if (launch_bgemm(g, &g2, ws, ws_cap, s)) return;
  launch_gemm(g, ws, ws_cap, s);
  GemmArgs h = g2;
  h.C = g.C;
  h.ldc = g.ldc;
  h.beta = 1.f;
  launch_gemm(h, ws, ws_cap, s);
}

// ------------------------------------------------------------- column sums ----
constexpr int COLSUM_SPLITS = 128;
__global__ void k_colsum1(const float* __restrict__ in, int64_t rows, int64_t cols, int64_t ld, float* __restrict__ ws) {
  const int64_t c = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (c >= cols) return;
  const int s = blockIdx.y;
  const int64_t chunk = (rows + COLSUM_SPLITS - 1) / COLSUM_SPLITS;
  const int64_t r0 = s * chunk, r1 = min(rows, r0 + chunk);
  float acc = 0.f;
  for (int64_t r = r0; r < r1; ++r) acc += in[r * ld + c];
  ws[s * cols + c] = acc;
}
// 64 columns per block; thread group q of four adds the partials q*S/4 ..
// (q+1)*S/4 - 1 in order, and the four group sums are added in group order.
__global__ __launch_bounds__(256) void k_colsum2(const float* __restrict__ ws, int64_t cols, float* out, float beta) {
  __shared__ float red[4][64];
  constexpr int PER = COLSUM_SPLITS / 4;
  const int q = threadIdx.x >> 6, cl = threadIdx.x & 63;
  const int64_t c = (int64_t)blockIdx.x * 64 + cl;
  float acc = 0.f;
  if (c < cols) {
#pragma unroll 16
    for (int s = q * PER; s < (q + 1) * PER; ++s) acc += ws[s * cols + c];
  }
  red[q][cl] = acc;
  __syncthreads();
  if (q == 0 && c < cols) {
    const float tot = ((red[0][cl] + red[1][cl]) + red[2][cl]) + red[3][cl];
    out[c] = (beta != 0.f) ? out[c] + tot : tot;
  }
}
// four columns per thread, eight rows in flight; the four waves of a block
// take consecutive quarters of the split's rows, and their sums are added in
// wave order
// (gridDim.y splits of the rows; with one, the sums go straight to out, added
// to it when beta is not 0)
__global__ __launch_bounds__(256) void k_colsum1v(const float* __restrict__ in, int64_t rows, int64_t cols, int64_t ld,
                                                  float* __restrict__ ws, float* __restrict__ out, float beta) {
  __shared__ float4 red[4][64];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t c = ((int64_t)blockIdx.x * 64 + lane) * 4;
  const int s = blockIdx.y;
  const int64_t chunk = (rows + gridDim.y - 1) / gridDim.y;
  const int64_t r0s = s * chunk, r1s = min(rows, r0s + chunk);
  const int64_t sub = (chunk + 3) / 4;
  const int64_t r0 = r0s + wave * sub, r1 = min(r1s, r0 + sub);
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  auto add = [&](const float4& v) {
    acc.x += v.x;
    acc.y += v.y;
    acc.z += v.z;
    acc.w += v.w;
  };
  if (c < cols) {
    int64_t r = r0;
    for (; r + 8 <= r1; r += 8) {
      float4 v[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) v[j] = *reinterpret_cast<const float4*>(in + (r + j) * ld + c);
#pragma unroll
      for (int j = 0; j < 8; ++j) add(v[j]);
    }
    for (; r < r1; ++r) add(*reinterpret_cast<const float4*>(in + r * ld + c));
  }
  red[wave][lane] = acc;
  __syncthreads();
  if (wave == 0 && c < cols) {
    float4 t = red[0][lane];
#pragma unroll
    for (int w = 1; w < 4; ++w) {
      const float4 v = red[w][lane];
      t.x += v.x;
      t.y += v.y;
      t.z += v.z;
      t.w += v.w;
    }
    if (gridDim.y > 1) {
      *reinterpret_cast<float4*>(ws + s * cols + c) = t;
    } else {
      float4* o = reinterpret_cast<float4*>(out + c);
      if (beta != 0.f) {
        const float4 u = *o;
        t = make_float4(u.x + t.x, u.y + t.y, u.z + t.z, u.w + t.w);
      }
      *o = t;
    }
  }
}
int64_t colsum_ws_floats(int64_t cols) { return COLSUM_SPLITS * cols; }
void launch_colsum(const float* in, int64_t rows, int64_t cols, int64_t ld, float* out, float beta, float* ws,
                   hipStream_t s) {
  const unsigned gx = (unsigned)((cols + 255) / 256);
  const bool vec = cols % 4 == 0 && ld % 4 == 0 && ((uintptr_t)in & 15) == 0;
  // few rows (sums over chunks of windows): one pass, each block over all rows
  if (vec && rows <= 512 && ((uintptr_t)out & 15) == 0) {
    hipLaunchKernelGGL(k_colsum1v, dim3((unsigned)((cols / 4 + 63) / 64), 1), dim3(256), 0, s, in, rows, cols, ld, ws,
                       out, beta);
    return;
  }
  if (vec)
    hipLaunchKernelGGL(k_colsum1v, dim3(gx, COLSUM_SPLITS), dim3(256), 0, s, in, rows, cols, ld, ws, out, beta);
  else
    hipLaunchKernelGGL(k_colsum1, dim3(gx, COLSUM_SPLITS), dim3(256), 0, s, in, rows, cols, ld, ws);
  hipLaunchKernelGGL(k_colsum2, dim3((unsigned)((cols + 63) / 64)), dim3(256), 0, s, ws, cols, out, beta);
}

// ------------------------------------------------------ head: dz of the CE ----
// dz[n] = (softmax(z[n]) - onehot(y[n])) / N for the mean cross-entropy in nats.
// One wave per window; each lane holds 4 of the 256 logits.
__global__ __launch_bounds__(256) void k_ce_grad(const float* __restrict__ z, const int32_t* __restrict__ tgt, int64_t N,
                                                 float* __restrict__ dz) {
  const int lane = threadIdx.x & 63;
  const int64_t n = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (n >= N) return;
  float v[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) v[i] = z[n * 256 + lane + 64 * i];
  float mx = fmaxf(fmaxf(v[0], v[1]), fmaxf(v[2], v[3]));
  for (int o = 32; o > 0; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o, 64));
  float ex[4], sm = 0.f;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    ex[i] = expf(v[i] - mx);
    sm += ex[i];
  }
  for (int o = 32; o > 0; o >>= 1) sm += __shfl_xor(sm, o, 64);
  const int y = tgt[n];
  const float fn = (float)N;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int c = lane + 64 * i;
    const float p = ex[i] / sm;
    dz[n * 256 + c] = (p - (c == y ? 1.f : 0.f)) / fn;
  }
}
void launch_ce_grad(const float* z, const int32_t* tgt, int64_t N, float* dz, hipStream_t s) {
  hipLaunchKernelGGL(k_ce_grad, dim3((unsigned)((N + 3) / 4)), dim3(256), 0, s, z, tgt, N, dz);
}

// -------------------------------------------------------------- elementwise ----
__global__ void k_gelu_fwd_round(const float* __restrict__ U, float* __restrict__ G, int64_t n, int round) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= n) return;
  const float g = gelu_f(U[i]);
  G[i] = round ? round_bf(g) : g;
}
void launch_gelu_fwd_round(const float* U, float* G, int64_t n, int round, hipStream_t s) {
  hipLaunchKernelGGL(k_gelu_fwd_round, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, U, G, n, round);
}
// (dU may be dG: each element is read before it is written, by one thread)
__global__ void k_gelu_bwd(const float* dG, const float* __restrict__ U, float* dU, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= n) return;
  dU[i] = dG[i] * gelu_grad_f(U[i]);
}
void launch_gelu_bwd(const float* dG, const float* U, float* dU, int64_t n, hipStream_t s) {
  hipLaunchKernelGGL(k_gelu_bwd, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, dG, U, dU, n);
}
// y[r][c] += x[r][c]
__global__ void k_add(float* __restrict__ y, const float* __restrict__ x, int64_t rows, int64_t cols, int64_t ldy,
                      int64_t ldx) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= rows * cols) return;
  const int64_t r = i / cols, c = i % cols;
  y[r * ldy + c] += x[r * ldx + c];
}
// the same, four columns per thread (cols, ldy, ldx multiples of 4, 16-byte aligned rows)
__global__ __launch_bounds__(256) void k_add4(float* __restrict__ y, const float* __restrict__ x, uint32_t rows,
                                              uint32_t cols4, int64_t ldy, int64_t ldx) {
  const uint32_t q = blockIdx.x * 256u + threadIdx.x;
  if (q >= rows * cols4) return;
  const uint32_t r = q / cols4, c = (q - r * cols4) * 4;
  float4* py = reinterpret_cast<float4*>(y + r * ldy + c);
  const float4 a = *py, b = *reinterpret_cast<const float4*>(x + r * ldx + c);
  *py = make_float4(a.x + b.x, a.y + b.y, a.z + b.z, a.w + b.w);
}
void launch_add(float* y, const float* x, int64_t rows, int64_t cols, int64_t ldy, int64_t ldx, hipStream_t s) {
  if (rows <= 0 || cols <= 0) return;
  if (cols % 4 == 0 && ldy % 4 == 0 && ldx % 4 == 0 && ((uintptr_t)y & 15) == 0 && ((uintptr_t)x & 15) == 0 &&
      rows * cols / 4 < ((int64_t)1 << 32)) {
    const int64_t n4 = rows * cols / 4;
    hipLaunchKernelGGL(k_add4, dim3((unsigned)((n4 + 255) / 256)), dim3(256), 0, s, y, x, (uint32_t)rows,
                       (uint32_t)(cols / 4), ldy, ldx);
  } else {
    hipLaunchKernelGGL(k_add, dim3((unsigned)((rows * cols + 255) / 256)), dim3(256), 0, s, y, x, rows, cols, ldy, ldx);
  }
}

// ------------------------------------------------------- attention backward ----
// Attention backward of the last query row (Eqs. 1-2).  A block takes one
// head of 4 (DH = 64) or 8 (DH = 32) consecutive windows, a wave (half a wave)
// per window and a lane per column: dA_u = dO_h . V_h[u] by shuffle sums over
// the head's lanes, dS = A (dA - sum_u A_u dA_u), dQ_h = scale sum_u dS_u
// K_h[u], dK_h[u] = scale dS_u q_h, dV_h[u] = A_u dO_h.  The block also adds
// its windows' dK and dV rows in a fixed order into part[chunk][0|1][u][col]:
// the sums over windows that the positional gradients need come from a column
// sum over the chunks (launch_colsum) instead of over every window's rows.
// part NULL: no sums (they come from the rank-one rows, launch_rank1_sums).
template <int DH>
__global__ __launch_bounds__(256) void k_attn_bwd2(const float* __restrict__ dO, const float* __restrict__ q,
                                                   const float* __restrict__ K, const float* __restrict__ V,
                                                   const float* __restrict__ A, int64_t N, int T, int D, int H,
                                                   float scale, int round_dO, float* __restrict__ dQ,
                                                   float* __restrict__ dK, float* __restrict__ dV,
                                                   float* __restrict__ part, float* __restrict__ dS) {
  constexpr int PW = 64 / DH;  // windows per wave
  constexpr int CH = 4 * PW;   // windows per block
  __shared__ float red[2][CH][8][DH];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int c = lane % DH, sub = lane / DH, slot = wave * PW + sub;
  const int h = blockIdx.x % H;
  const int64_t ch = blockIdx.x / H;
  const int col = h * DH + c;
  const int64_t n = ch * CH + slot;
  const bool live = n < N;
  const int64_t nn = live ? n : ch * CH;  // dead slots redo the chunk's first window and store nothing
  float o = dO[nn * D + col];
  // (bf16 rounding by the hardware conversion: round to nearest even, no branch)
  if (round_dO) o = __uint_as_float(pack_bf16x2(o, 0.f) << 16);
  // every row of V and K first (all loads in flight together)
  float vr[8], kr[8], a[8], dA[8];
#pragma unroll
  for (int u = 0; u < 8; ++u) {
    vr[u] = u < T ? V[(nn * T + u) * D + col] : 0.f;
    kr[u] = u < T ? K[(nn * T + u) * D + col] : 0.f;
    a[u] = u < T ? A[(nn * H + h) * T + u] : 0.f;
  }
  const float qv = q[nn * D + col];
  float tot = 0.f;
#pragma unroll
  for (int u = 0; u < 8; ++u) {
    if (u < T) {
      float x = o * vr[u];
#pragma unroll
      for (int off = 1; off < DH; off <<= 1) x += __shfl_xor(x, off, 64);
      dA[u] = x;
      tot = fmaf(a[u], x, tot);
    }
  }
  float dq = 0.f;
#pragma unroll
  for (int u = 0; u < 8; ++u) {
    if (u < T) {
      const float ds = a[u] * (dA[u] - tot);
      if (dS && live && c == 0) dS[(nn * H + h) * T + u] = ds;
      dq = fmaf(ds, kr[u], dq);
      const float dk = (ds * qv) * scale, dv = a[u] * o;
      if (live && dK) {
        dK[(nn * T + u) * D + col] = dk;
        dV[(nn * T + u) * D + col] = dv;
      }
      if (part) {
        red[0][slot][u][c] = live ? dk : 0.f;
        red[1][slot][u][c] = live ? dv : 0.f;
      }
    }
  }
  if (live) dQ[nn * D + col] = dq * scale;
  if (!part) return;  // (uniform over the grid)
  __syncthreads();
  for (int i = threadIdx.x; i < 2 * T * DH; i += 256) {
    const int which = i / (T * DH), u = (i / DH) % T, cc = i % DH;
    float v = 0.f;
#pragma unroll
    for (int k = 0; k < CH; ++k) v += red[which][k][u][cc];
    part[((ch * 2 + which) * T + u) * D + h * DH + cc] = v;
  }
}

// The same backward for the rank-one path (no dK, dV rows, no window sums, so
// no q): one wave per window, lane l holding columns CPL l .. CPL l + CPL - 1 (CPL = D / 64,
// one head's DH / CPL lanes consecutive), so that every row of K and V comes in
// CPL-float vector loads, all T rows of both first.  dA_u by a lane sum and a
// shuffle tree over the head's lanes; dS and dQ as in k_attn_bwd2.
template <int D, int DH, int T, bool NTL>
__global__ __launch_bounds__(256) void k_attn_bwd_r1(const float* __restrict__ dO, const float* __restrict__ K,
                                                     const float* __restrict__ V,
                                                     const float* __restrict__ A, int64_t N, float scale,
                                                     int round_dO, float* __restrict__ dQ, float* __restrict__ dS) {
  constexpr int CPL = D / 64, LPH = DH / CPL, H = D / DH;
  static_assert(CPL == 2 || CPL == 4 || CPL == 8, "columns per lane");
  static_assert(LPH >= 1 && (LPH & (LPH - 1)) == 0 && LPH <= 64, "lanes per head");
  typedef float __attribute__((ext_vector_type(CPL == 2 ? 2 : 4))) vec;
  constexpr int NV = CPL == 8 ? 2 : 1;  // vector loads per row
  constexpr int VW = CPL / NV;          // floats per vector load
  const int lane = threadIdx.x & 63;
  const int64_t n = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (n >= N) return;  // (whole waves)
  const int c0 = lane * CPL, h = c0 / DH;
  float kr[T][CPL], vr[T][CPL], o[CPL], a[T];
  // NTL: K and V larger than the last-level cache, streamed past it (they are
  // read once), the V rows first (dA needs them alone), then K's, so that the
  // dot products of dA run while the K rows arrive; otherwise row by row
  auto ld = [](const float* p) {
    if constexpr (NTL)
      return __builtin_nontemporal_load(reinterpret_cast<const vec*>(p));
    else
      return *reinterpret_cast<const vec*>(p);
  };
#pragma unroll
  for (int u = 0; u < T; ++u)
#pragma unroll
    for (int e = 0; e < NV; ++e) {
      const vec x = ld(V + (n * T + u) * D + c0 + e * VW);
#pragma unroll
      for (int i = 0; i < VW; ++i) vr[u][e * VW + i] = x[i];
      if constexpr (!NTL) {
        const vec y = ld(K + (n * T + u) * D + c0 + e * VW);
#pragma unroll
        for (int i = 0; i < VW; ++i) kr[u][e * VW + i] = y[i];
      }
    }
#pragma unroll
  for (int e = 0; e < NV; ++e) {
    const vec x = *reinterpret_cast<const vec*>(dO + n * D + c0 + e * VW);
#pragma unroll
    for (int i = 0; i < VW; ++i) o[e * VW + i] = x[i];
  }
#pragma unroll
  for (int u = 0; u < T; u += 4) {
    const float4 x = *reinterpret_cast<const float4*>(A + (n * H + h) * T + u);
    a[u] = x.x; a[u + 1] = x.y; a[u + 2] = x.z; a[u + 3] = x.w;
  }
  if constexpr (NTL) {
#pragma unroll
    for (int u = 0; u < T; ++u)
#pragma unroll
      for (int e = 0; e < NV; ++e) {
        const vec y = ld(K + (n * T + u) * D + c0 + e * VW);
#pragma unroll
        for (int i = 0; i < VW; ++i) kr[u][e * VW + i] = y[i];
      }
  }
  // (bf16 rounding by the hardware conversion: round to nearest even, no branch)
  if (round_dO) {
#pragma unroll
    for (int i = 0; i < CPL; ++i) o[i] = __uint_as_float(pack_bf16x2(o[i], 0.f) << 16);
  }
  float dA[T], tot = 0.f;
#pragma unroll
  for (int u = 0; u < T; ++u) {
    float x = 0.f;
#pragma unroll
    for (int i = 0; i < CPL; ++i) x = fmaf(o[i], vr[u][i], x);
#pragma unroll
    for (int off = 1; off < LPH; off <<= 1) x += __shfl_xor(x, off, 64);
    dA[u] = x;
    tot = fmaf(a[u], x, tot);
  }
  float dq[CPL];
#pragma unroll
  for (int i = 0; i < CPL; ++i) dq[i] = 0.f;
  float ds[T];
#pragma unroll
  for (int u = 0; u < T; ++u) {
    ds[u] = a[u] * (dA[u] - tot);
#pragma unroll
    for (int i = 0; i < CPL; ++i) dq[i] = fmaf(ds[u], kr[u][i], dq[i]);
  }
#pragma unroll
  for (int e = 0; e < NV; ++e) {
    vec x;
#pragma unroll
    for (int i = 0; i < VW; ++i) x[i] = dq[e * VW + i] * scale;
    *reinterpret_cast<vec*>(dQ + n * D + c0 + e * VW) = x;
  }
  if ((lane & (LPH - 1)) == 0) {
#pragma unroll
    for (int u = 0; u < T; u += 4)
      *reinterpret_cast<float4*>(dS + (n * H + h) * T + u) = make_float4(ds[u], ds[u + 1], ds[u + 2], ds[u + 3]);
  }
}

int64_t attn_bwd_chunks(int64_t N, int D, int H) { return (N + 4 * (64 / (D / H)) - 1) / (4 * (64 / (D / H))); }

int64_t attn_bwd_part_floats(int64_t N, int T, int D, int H) { return attn_bwd_chunks(N, D, H) * 2 * T * D; }

void launch_attn_bwd(const float* dO, const float* q, const float* K, const float* V, const float* A, int64_t N, int T,
                     int D, int H, float scale, int round_dO, float* dQ, float* dK, float* dV, float* part,
                     float* colsums, float* cws, hipStream_t s, float* dS) {
  const int DH = D / H;
  if (!dK && !dV && !part && dS && N > 0 && (T == 4 || T == 8)) {
    // the rank-one path: one wave per window; K and V streamed when together
    // larger than 128 MiB (half the last-level cache)
    const dim3 g4((unsigned)((N + 3) / 4));
    const bool ntl = (int64_t)2 * N * T * D * 4 > ((int64_t)128 << 20);
#define TRACE_ABR1(D_, DH_, T_)                                                                                    \
  if (D == D_ && DH == DH_ && T == T_) {                                                                           \
    if (ntl)                                                                                                       \
      hipLaunchKernelGGL((k_attn_bwd_r1<D_, DH_, T_, true>), g4, dim3(256), 0, s, dO, K, V, A, N, scale, round_dO, \
                         dQ, dS);                                                                                  \
    else                                                                                                           \
      hipLaunchKernelGGL((k_attn_bwd_r1<D_, DH_, T_, false>), g4, dim3(256), 0, s, dO, K, V, A, N, scale,         \
                         round_dO, dQ, dS);                                                                        \
    return;                                                                                                        \
  }
    TRACE_ABR1(128, 32, 4) TRACE_ABR1(128, 32, 8) TRACE_ABR1(128, 64, 4) TRACE_ABR1(128, 64, 8)
    TRACE_ABR1(256, 32, 4) TRACE_ABR1(256, 32, 8) TRACE_ABR1(256, 64, 4) TRACE_ABR1(256, 64, 8)
    TRACE_ABR1(512, 64, 4) TRACE_ABR1(512, 64, 8)
#undef TRACE_ABR1
  }
  const int64_t chunks = attn_bwd_chunks(N, D, H);
  const dim3 grid((unsigned)(chunks * H));
  if (DH == 32)
    hipLaunchKernelGGL(k_attn_bwd2<32>, grid, dim3(256), 0, s, dO, q, K, V, A, N, T, D, H, scale, round_dO, dQ, dK,
                       dV, part, dS);
  else
    hipLaunchKernelGGL(k_attn_bwd2<64>, grid, dim3(256), 0, s, dO, q, K, V, A, N, T, D, H, scale, round_dO, dQ, dK,
                       dV, part, dS);
  if (part) launch_colsum(part, chunks, (int64_t)2 * T * D, (int64_t)2 * T * D, colsums, 0.f, cws, s);
}

// Sums over windows of the last query row's key and value gradients from their
// rank-one rows, for the positional parts of the weight gradients and of the
// positional table (the same values k_attn_bwd2 sums), with the sums of dQ and
// dY0 beside them:
//   sK[t][j] = sum_n (dS[n][h][t] q[n][j]) scale,  sV[t][j] = sum_n A[n][h][t] bf(dO[n][j]),
//   sQ[j] = sum_n dQ[n][j],  sY[j] = sum_n dY0[n][j],  h = j / DH.
// A block takes 64 columns of a chunk of RS_CW windows; its wave s the windows
// s, s + 8, ... (half of them at a time, every load first), the eight waves'
// sums are added in wave order into part[chunk][2 T + 2][D] (rows sK, sV, sQ,
// sY), and a column sum over the chunks follows (launch_colsum).
constexpr int RS_CW = 64;
constexpr int RS_W = 8;  // waves per block
constexpr int RS_B = RS_CW / (2 * RS_W);  // windows per wave and batch (two batches: 164 registers for one)
template <int T>
__global__ __launch_bounds__(64 * RS_W) void k_rank1_sums(const float* __restrict__ dS, const float* __restrict__ q,
                                                          const float* __restrict__ A, const float* __restrict__ dO,
                                                          const float* __restrict__ dQ, const float* __restrict__ dY0,
                                                          int64_t N, int D, int H, int dsh, float scale,
                                                          int round_dO, float* __restrict__ part) {
  constexpr int NR = 2 * T + 2;  // rows of sums
  __shared__ float red[RS_W][NR][64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int j = blockIdx.y * 64 + lane, h = j >> dsh;
  const int64_t c = blockIdx.x, n0 = c * RS_CW;
  const int nw = (int)min<int64_t>(RS_CW, N - n0);
  float sk[T], sv[T], sq = 0.f, sy = 0.f;
#pragma unroll
  for (int t = 0; t < T; ++t) sk[t] = sv[t] = 0.f;
#pragma unroll
  for (int i0 = 0; i0 < RS_CW; i0 += RS_B * RS_W) {
    float qv[RS_B], ov[RS_B], gq[RS_B], gy[RS_B], ds[RS_B][T], aa[RS_B][T];
#pragma unroll
    for (int u = 0; u < RS_B; ++u) {
      const int64_t n = n0 + min(i0 + RS_W * u + wave, nw - 1);  // clamped; the window is not added
      qv[u] = q[n * D + j];
      ov[u] = dO[n * D + j];
      gq[u] = dQ[n * D + j];
      gy[u] = dY0[n * D + j];
#pragma unroll
      for (int t = 0; t < T; t += 4) {
        const float4 x = *reinterpret_cast<const float4*>(dS + (n * H + h) * T + t);
        const float4 y = *reinterpret_cast<const float4*>(A + (n * H + h) * T + t);
        ds[u][t] = x.x; ds[u][t + 1] = x.y; ds[u][t + 2] = x.z; ds[u][t + 3] = x.w;
        aa[u][t] = y.x; aa[u][t + 1] = y.y; aa[u][t + 2] = y.z; aa[u][t + 3] = y.w;
      }
    }
#pragma unroll
    for (int u = 0; u < RS_B; ++u) {
      if (i0 + RS_W * u + wave < nw) {
        float o = ov[u];
        if (round_dO) o = __uint_as_float(pack_bf16x2(o, 0.f) << 16);
#pragma unroll
        for (int t = 0; t < T; ++t) {
          sk[t] += (ds[u][t] * qv[u]) * scale;
          sv[t] += aa[u][t] * o;
        }
        sq += gq[u];
        sy += gy[u];
      }
    }
  }
#pragma unroll
  for (int t = 0; t < T; ++t) {
    red[wave][t][lane] = sk[t];
    red[wave][T + t][lane] = sv[t];
  }
  red[wave][2 * T][lane] = sq;
  red[wave][2 * T + 1][lane] = sy;
  __syncthreads();
  for (int i = threadIdx.x; i < NR * 64; i += 64 * RS_W) {
    const int r = i / 64, jj = i % 64;
    float v = red[0][r][jj];
#pragma unroll
    for (int w = 1; w < RS_W; ++w) v += red[w][r][jj];
    part[(c * NR + r) * D + blockIdx.y * 64 + jj] = v;
  }
}

int64_t rank1_sums_part_floats(int64_t N, int T, int D) { return (N + RS_CW - 1) / RS_CW * (2 * T + 2) * D; }

bool launch_rank1_sums(const float* dS, const float* q, const float* A, const float* dO, const float* dQ,
                       const float* dY0, int64_t N, int T, int D, int H, float scale, int round_dO, float* part,
                       float* colsums, float* cws, hipStream_t s) {
  const int DH = D / H;
  if (D % 64 != 0 || (DH & (DH - 1)) != 0 || (T != 4 && T != 8)) return false;
  const int64_t cols = (int64_t)(2 * T + 2) * D;
  if (N <= 0) {
    launch_zero(reinterpret_cast<uint32_t*>(colsums), cols, s);
    return true;
  }
  int dsh = 0;
  while ((1 << dsh) < DH) ++dsh;
  const int64_t chunks = (N + RS_CW - 1) / RS_CW;
  const dim3 grid((unsigned)chunks, (unsigned)(D / 64));
  if (T == 8)
    hipLaunchKernelGGL(k_rank1_sums<8>, grid, dim3(64 * RS_W), 0, s, dS, q, A, dO, dQ, dY0, N, D, H, dsh, scale,
                       round_dO, part);
  else
    hipLaunchKernelGGL(k_rank1_sums<4>, grid, dim3(64 * RS_W), 0, s, dS, q, A, dO, dQ, dY0, N, D, H, dsh, scale,
                       round_dO, part);
  launch_colsum(part, chunks, cols, cols, colsums, 0.f, cws, s);
  return true;
}

// Input gradient of the tokens through the keys and values, bf16 models:
// dX[n][t] = sum_h dK_h[n][t] . Wk_h^T + dV_h[n][t] . Wv_h^T with the rank-one
// rows dK_h[n][t] = dS[n][h][t] (scale q_h[n]) and dV_h[n][t] = A[n][h][t]
// bf(dO_h[n]), so that
//   dX[n][t] = sum_h dS[n][h][t] QK[n][h] + A[n][h][t] OV[n][h],
//   QK[n][h] = Wk_h . (scale q_h[n]),  OV[n][h] = Wv_h . bf(dO_h[n]),
// where Wk_h is the head's D x DH column block (weights rounded to bf16 as the
// product's operands).  QK and OV are formed on the matrix cores (scale q in
// hi + lo bf16 parts, dO exact in bf16), 2 D DH flops each per window and head
// instead of 2 T D DH for the products over every token row; the T-fold
// combination runs on the vector ALUs.  dY0 (the residual's gradient) is added
// to the last token.
// One block of 8 waves per 16 windows (the 16 columns of the B operand); wave
// w owns features [w D/8, (w+1) D/8), its accumulators acc[t][f] holding
// features w D/8 + 16 f + 4 lg + r of window n0 + lc.  The block first stages
// its windows' B operands (scale q as hi and lo, dO, in bf16; unit u of row m
// at u ^ (m & 15)) and their score gradients and weights in LDS with coalesced
// loads; the weights come as fragment-packed copies of Wk^T and Wv^T, one
// contiguous 16-byte load per lane and fragment.  dX is stored token row by
// token row, the row's fragments back to back (each store covers 64 bytes of a
// row; issued together, the halves of a 128-byte line reach the L2 together
// and are written once: non-temporal stores wrote 1.37 times the bytes).
template <int D, int DH, int T>
__global__ __launch_bounds__(512) void k_dx_rank1(const float* __restrict__ q, const float* __restrict__ dO,
                                                  const float* __restrict__ dS, const float* __restrict__ A,
                                                  const uint4* __restrict__ WkT, const uint4* __restrict__ WvT,
                                                  const float* __restrict__ dY0, int64_t N, float scale,
                                                  float* __restrict__ dX) {
  constexpr int H = D / DH, KS = DH / 32, NF = D / 128, NB = D / 16;
  constexpr int RU = D / 8;          // 16-byte units per staged row
  constexpr int SST = H * T + 4;     // floats per staged score row (padded: conflict-free lane reads)
  static_assert(D % 128 == 0 && DH % 32 == 0 && T <= 8 && T % 4 == 0, "shape");
  typedef Mma<true> M;
  __shared__ uint4 Bq[3][16 * RU];   // scale q hi, scale q lo, dO
  __shared__ __align__(16) float Sds[2][16 * SST];  // dS, A
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, lg = lane >> 4, lc = lane & 15;
  const int64_t n0 = (int64_t)blockIdx.x * 16;
  const int nwin = (int)min<int64_t>(16, N - n0);
  // stage: rows n0 .. n0 + 15 of q and dO (four floats per thread and step),
  // of dS and A (rows past N: zeros)
  for (int i = tid; i < 16 * D / 4; i += 512) {
    const int m = i / (D / 4), c4 = i - m * (D / 4);
    float4 v = make_float4(0.f, 0.f, 0.f, 0.f), o = v;
    if (m < nwin) {
      v = *reinterpret_cast<const float4*>(q + (n0 + m) * D + 4 * c4);
      o = *reinterpret_cast<const float4*>(dO + (n0 + m) * D + 4 * c4);
    }
    v.x *= scale;
    v.y *= scale;
    v.z *= scale;
    v.w *= scale;
    const uint32_t h0 = pack_bf16x2(v.x, v.y), h1 = pack_bf16x2(v.z, v.w);
    const uint32_t l0 = pack_bf16x2(v.x - __uint_as_float(h0 << 16), v.y - __uint_as_float(h0 & 0xffff0000u));
    const uint32_t l1 = pack_bf16x2(v.z - __uint_as_float(h1 << 16), v.w - __uint_as_float(h1 & 0xffff0000u));
    const int off = (m * RU + ((c4 >> 1) ^ (m & 15))) * 16 + 8 * (c4 & 1);  // bytes
    *reinterpret_cast<uint2*>(reinterpret_cast<unsigned char*>(Bq[0]) + off) = make_uint2(h0, h1);
    *reinterpret_cast<uint2*>(reinterpret_cast<unsigned char*>(Bq[1]) + off) = make_uint2(l0, l1);
    *reinterpret_cast<uint2*>(reinterpret_cast<unsigned char*>(Bq[2]) + off) =
        make_uint2(pack_bf16x2(o.x, o.y), pack_bf16x2(o.z, o.w));
  }
  for (int i = tid; i < 2 * 16 * H * T; i += 512) {
    const int which = i / (16 * H * T), j = i - which * (16 * H * T), m = j / (H * T), c = j - m * (H * T);
    Sds[which][m * SST + c] = m < nwin ? (which ? A : dS)[(n0 + m) * H * T + c] : 0.f;
  }
  __syncthreads();

  const int d0 = wave * (D / 8);
  float acc[T][NF][4];
#pragma unroll
  for (int t = 0; t < T; ++t)
#pragma unroll
    for (int f = 0; f < NF; ++f)
#pragma unroll
      for (int r = 0; r < 4; ++r) acc[t][f][r] = 0.f;
  for (int h = 0; h < H; ++h) {
    // A fragments (rows d0 + 16 f + lc, k = 32 (h KS + ks) + 8 lg + j): fragment
    // (ks', nb) of the packed copy at ((ks' NB + nb) 64 + lane)
    uint4 ak[NF][KS], av[NF][KS];
#pragma unroll
    for (int f = 0; f < NF; ++f)
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const int64_t fi = ((int64_t)(h * KS + ks) * NB + d0 / 16 + f) * 64 + lane;
        ak[f][ks] = WkT[fi];
        av[f][ks] = WvT[fi];
      }
    uint4 bqh[KS], bql[KS], bo[KS];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const int u = ((h * KS + ks) * 4 + lg) ^ lc;
      bqh[ks] = Bq[0][lc * RU + u];
      bql[ks] = Bq[1][lc * RU + u];
      bo[ks] = Bq[2][lc * RU + u];
    }
    float ds[T], aa[T];
#pragma unroll
    for (int t = 0; t < T; t += 4) {
      const float4 x = *reinterpret_cast<const float4*>(&Sds[0][lc * SST + h * T + t]);
      const float4 y = *reinterpret_cast<const float4*>(&Sds[1][lc * SST + h * T + t]);
      ds[t] = x.x; ds[t + 1] = x.y; ds[t + 2] = x.z; ds[t + 3] = x.w;
      aa[t] = y.x; aa[t + 1] = y.y; aa[t + 2] = y.z; aa[t + 3] = y.w;
    }
#pragma unroll
    for (int f = 0; f < NF; ++f) {
      f32x4 qk = f32x4{0.f, 0.f, 0.f, 0.f}, ov = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        M::run(qk, ak[f][ks], bqh[ks]);
        M::run(qk, ak[f][ks], bql[ks]);
        M::run(ov, av[f][ks], bo[ks]);
      }
#pragma unroll
      for (int t = 0; t < T; ++t)
#pragma unroll
        for (int r = 0; r < 4; ++r) acc[t][f][r] = fmaf(aa[t], ov[r], fmaf(ds[t], qk[r], acc[t][f][r]));
    }
  }
  if (lc >= nwin) return;
  const int64_t n = n0 + lc;
#pragma unroll
  for (int f = 0; f < NF; ++f) {
    const int d = d0 + 16 * f + 4 * lg;
    const float4 y = *reinterpret_cast<const float4*>(dY0 + n * D + d);
    acc[T - 1][f][0] += y.x;
    acc[T - 1][f][1] += y.y;
    acc[T - 1][f][2] += y.z;
    acc[T - 1][f][3] += y.w;
  }
#pragma unroll
  for (int t = 0; t < T; ++t)
#pragma unroll
    for (int f = 0; f < NF; ++f) {
      const int d = d0 + 16 * f + 4 * lg;
      const f32x4 v = f32x4{acc[t][f][0], acc[t][f][1], acc[t][f][2], acc[t][f][3]};
      *reinterpret_cast<f32x4*>(dX + (n * T + t) * D + d) = v;
    }
}

template <int D, int DH, int T>
static void launch_dx_rank1_t(const float* q, const float* dO, const float* dS, const float* A, const uint4* WkT,
                              const uint4* WvT, const float* dY0, int64_t N, float scale, float* dX, hipStream_t s) {
  hipLaunchKernelGGL((k_dx_rank1<D, DH, T>), dim3((unsigned)((N + 15) / 16)), dim3(512), 0, s, q, dO, dS, A, WkT, WvT,
                     dY0, N, scale, dX);
}

bool dx_rank1_built(int T, int D, int H) {
  const int DH = D / H;
  return (D == 128 || D == 256 || (D == 512 && DH == 64)) && (DH == 32 || DH == 64) && (T == 4 || T == 8);
}

bool launch_dx_rank1(const float* q, const float* dO, const float* dS, const float* A, const uint4* WkT,
                     const uint4* WvT, const float* dY0, int64_t N, int T, int D, int H, float scale, float* dX,
                     hipStream_t s) {
  if (N <= 0) return true;
  const int DH = D / H;
#define TRACE_DXR(D_, DH_, T_)                                                                      \
  if (D == D_ && DH == DH_ && T == T_) {                                                           \
    launch_dx_rank1_t<D_, DH_, T_>(q, dO, dS, A, WkT, WvT, dY0, N, scale, dX, s);                  \
    return true;                                                                                   \
  }
  TRACE_DXR(128, 32, 4) TRACE_DXR(128, 32, 8) TRACE_DXR(128, 64, 4) TRACE_DXR(128, 64, 8)
  TRACE_DXR(256, 32, 4) TRACE_DXR(256, 32, 8) TRACE_DXR(256, 64, 4) TRACE_DXR(256, 64, 8)
  TRACE_DXR(512, 64, 4) TRACE_DXR(512, 64, 8)
#undef TRACE_DXR
  return false;
}

// Weight gradients of the key and value projections (bf16 models, the rank-one
// rows of the last query row): with the token rows X[n][t] (byte-embedding part)
// and, per window n and head h,
//   ZK_h[n] = sum_t dS[n][h][t] X[n][t],   ZV_h[n] = sum_t A[n][h][t] X[n][t],
// the head-h columns of the gradients are
//   dWk[:, h] = sum_n ZK_h[n]^T (scale q_h[n]),   dWv[:, h] = sum_n ZV_h[n]^T bf(dO_h[n]),
// the same sums as X^T dK and X^T dV over every token row with T times fewer
// products.  Block: 32 rows d of the key or the value gradient over one range
// of windows, in tiles of 32 windows; H waves.  Per tile, both products run on
// v_mfma_f32_16x16x32_bf16:
//  1. Z^T = X^T Cbd: rows d, k = (window w, token t) over 32 / T windows per
//     k-step, columns (w', h) of 16 / H windows; Cbd(w t, w' h) = C[w][h][t]
//     where w = w', 0 elsewhere (block diagonal, C = dS or A as bf16 hi + lo,
//     packed as fragments by k_kv_pack).  X (the tokens' rows, or gathered
//     here from the window bytes and the embedding copy) is staged in LDS
//     transposed (rows d, k contiguous), double-buffered, so that a lane's A
//     fragment is one 16-byte read; the k-steps are dealt to the waves.  Z
//     goes to LDS as fp32, rows (h, d) of the tile's 32 windows.
//  2. wave h: dW[d][h DH + j] += sum_w Z_h[w][d] B[w][j], Z as bf16 hi + lo,
//     B = q as hi + lo (three products; the scale applied to the sums) or
//     bf(dO), exact (two), packed as fragments by k_kv_pack.  Fragment row m of
//     d-fragment f is d = 16 f + m, column c of j-fragment jf is
//     j = h DH + NJF c + jf.
// The next tile's fragments are loaded while the current one is used.
// Windows past the range have zero coefficients, so zero Z (their rows are read
// clamped).  Partial sums of the window range z go to part[z][kv][d][j]
// (kv 0: key, 1: value), summed by the split-K reduce.
constexpr int KVW_DC = 32, KVW_NT = 32;

template <int T, int H>
struct KvwLds {
  static constexpr int XR = KVW_NT * T + 8;   // bf16 per staged row d (k = w T + t) + 16 bytes of padding
  static constexpr int ZR = KVW_NT + 4;       // floats per Z row (h, d) + padding
  static constexpr int ZH = KVW_DC * ZR + 4;  // floats per head + padding
  uint16_t xt[2][KVW_DC * XR];
  float zs[H * ZH];
};

// bf16 hi + lo of eight values
__device__ __forceinline__ void kvw_split8(const float (&v)[8], uint4& hi, uint4& lo) {
  uint32_t a[4], b[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    a[i] = pack_bf16x2(v[2 * i], v[2 * i + 1]);
    b[i] = pack_bf16x2(v[2 * i] - __uint_as_float(a[i] << 16), v[2 * i + 1] - __uint_as_float(a[i] & 0xffff0000u));
  }
  hi = make_uint4(a[0], a[1], a[2], a[3]);
  lo = make_uint4(b[0], b[1], b[2], b[3]);
}

template <int T, int DH, int H, bool VAL>
__device__ __forceinline__ void kv_wgrad_body(KvwLds<T, H>& sm, const uint16_t* __restrict__ X,
                                              const uint8_t* __restrict__ win, const uint16_t* __restrict__ E,
                                              int e, int gw, const uint4* __restrict__ Cp,
                                              const uint4* __restrict__ Bp, int N, int nps, float bscale,
                                              float* __restrict__ part, int d0, int z, int S) {
  constexpr int D = H * DH, NJF = DH / 16, NTH = 64 * H;
  constexpr int XR = KvwLds<T, H>::XR, ZR = KvwLds<T, H>::ZR, ZH = KvwLds<T, H>::ZH;
  constexpr int NKS = KVW_NT * T / 32;  // k-steps of the first product per tile
  constexpr int WPC = 16 / H;           // windows per column block of Z^T
  constexpr int NCB = 32 / T / WPC;     // column blocks per k-step
  constexpr int NSU = KVW_NT * T / 8 * (KVW_DC / 8);  // staging units (8 k x 8 d)
  static_assert(NJF == 2 || NJF == 4, "head width");
  static_assert(NCB >= 1 && NSU <= NTH, "tile shape");
  const int h = threadIdx.x >> 6, l = threadIdx.x & 63, g = l >> 4, m = l & 15;
  const int nb = z * nps, ne = min(N, nb + nps);
  const int ntiles = (ne - nb + KVW_NT - 1) / KVW_NT;
  const bool stager = threadIdx.x < NSU;
  const int so = threadIdx.x >> 2, sp = threadIdx.x & 3;  // staging unit: k-octet so, d-octet sp

  // X of tile k, unit (so, sp): rows k = 8 so + i of d0 + 8 sp .. + 7, clamped
  // (32-bit element offsets: N T D < 2^30).  With win: gathered here, token
  // (n, t) columns c .. c + 7 being E[win[(n T + t) gw + c / e]][c % e ..] (gw
  // bytes per token, e a multiple of 8), all byte loads first
  uint4 xr[8];
  const int xc = d0 + 8 * sp, xj = win ? xc / e : 0, xcc = win ? xc - xj * e : 0;
  auto load = [&](int k) {
    if (!stager) return;
    const int n0 = nb + k * KVW_NT;
    if (win) {
      int by[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int kk = 8 * so + i, n = min(n0 + kk / T, N - 1), t = kk % T;
        by[i] = win[(uint32_t)(n * T + t) * gw + xj];
      }
#pragma unroll
      for (int i = 0; i < 8; ++i) xr[i] = *reinterpret_cast<const uint4*>(E + by[i] * e + xcc);
    } else {
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int kk = 8 * so + i, n = min(n0 + kk / T, N - 1), t = kk % T;
        xr[i] = *reinterpret_cast<const uint4*>(X + ((uint32_t)(n * T + t) * D + xc));
      }
    }
  };
  // transposed: row d = 8 sp + e holds k = 8 so .. + 7 (one 16-byte write)
  auto put = [&](int b) {
    if (!stager) return;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      uint32_t w[4];
#pragma unroll
      for (int a = 0; a < 4; ++a) {
        const uint32_t lo = (&xr[2 * a].x)[e >> 1], hi = (&xr[2 * a + 1].x)[e >> 1];
        w[a] = (e & 1) ? ((lo >> 16) | (hi & 0xffff0000u)) : ((lo & 0xffffu) | (hi << 16));
      }
      *reinterpret_cast<uint4*>(&sm.xt[b][(8 * sp + e) * XR + 8 * so]) = make_uint4(w[0], w[1], w[2], w[3]);
    }
  };
  // packed fragments of tile k (k_kv_pack): the first product's B (Cbd, hi and
  // lo) for this wave's k-steps, the second product's B (V: hi and lo for the
  // key, hi for the value)
  constexpr int NSI = (NKS + H - 1) / H, NBS = VAL ? 1 : 2;
  const int tile0 = nb / KVW_NT;
  auto loadF = [&](uint4 (&cf)[NSI][NCB][2], uint4 (&bf)[NJF][NBS], int k) {
    const int64_t tl = tile0 + k;
#pragma unroll
    for (int si = 0; si < NSI; ++si) {
      const int ks = min(h + si * H, NKS - 1);
#pragma unroll
      for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
        for (int e = 0; e < 2; ++e) cf[si][cb][e] = Cp[(((tl * NKS + ks) * NCB + cb) * 2 + e) * 64 + l];
    }
#pragma unroll
    for (int jf = 0; jf < NJF; ++jf)
#pragma unroll
      for (int e = 0; e < NBS; ++e) bf[jf][e] = Bp[(((tl * H + h) * NJF + jf) * NBS + e) * 64 + l];
  };

  f32x4 acc[2][NJF];
#pragma unroll
  for (int f = 0; f < 2; ++f)
#pragma unroll
    for (int jf = 0; jf < NJF; ++jf) acc[f][jf] = f32x4{0.f, 0.f, 0.f, 0.f};

  uint4 cf[NSI][NCB][2], bf[NJF][NBS];
  if (ntiles > 0) {
    load(0);
    loadF(cf, bf, 0);
    put(0);
  }
  __syncthreads();
#pragma unroll 1
  for (int k = 0; k < ntiles; ++k) {
    const int b = k & 1;
    // the next tile's fragments (clamped past the last tile: the pack has
    // every tile of the product)
    if (k + 1 < ntiles) load(k + 1);
    uint4 cn[NSI][NCB][2], bn[NJF][NBS];
    loadF(cn, bn, min(k + 1, ntiles - 1));
    // first product, k-steps ks = wave, wave + H, ..
#pragma unroll
    for (int si = 0; si < NSI; ++si) {
      const int ks = h + si * H;
      if (ks < NKS) {
#pragma unroll
        for (int f = 0; f < 2; ++f) {
          const uint4 xa = *reinterpret_cast<const uint4*>(&sm.xt[b][(16 * f + m) * XR + 32 * ks + 8 * g]);
#pragma unroll
          for (int cb = 0; cb < NCB; ++cb) {
            f32x4 o = f32x4{0.f, 0.f, 0.f, 0.f};
            Mma<true>::run(o, xa, cf[si][cb][0]);
            Mma<true>::run(o, xa, cf[si][cb][1]);
            // o[r]: Z[w][hh][d = 16 f + 4 g + r], w = 32 ks / T + cb WPC + m / H (in the tile)
            const int w = 32 * ks / T + cb * WPC + m / H, hh = m % H;
#pragma unroll
            for (int r = 0; r < 4; ++r) sm.zs[hh * ZH + (16 * f + 4 * g + r) * ZR + w] = o[r];
          }
        }
      }
    }
    __syncthreads();
    // second product, wave h: Z_h rows 16 f + m, windows 8 g + j
    uint4 zh[2], zl[2];
#pragma unroll
    for (int f = 0; f < 2; ++f) {
      const float* zp = &sm.zs[h * ZH + (16 * f + m) * ZR + 8 * g];
      const float4 a = *reinterpret_cast<const float4*>(zp), c = *reinterpret_cast<const float4*>(zp + 4);
      const float v[8] = {a.x, a.y, a.z, a.w, c.x, c.y, c.z, c.w};
      kvw_split8(v, zh[f], zl[f]);
    }
#pragma unroll
    for (int jf = 0; jf < NJF; ++jf)
#pragma unroll
      for (int f = 0; f < 2; ++f) {
        Mma<true>::run(acc[f][jf], zh[f], bf[jf][0]);
        Mma<true>::run(acc[f][jf], zl[f], bf[jf][0]);
        if constexpr (!VAL) Mma<true>::run(acc[f][jf], zh[f], bf[jf][NBS - 1]);
      }
    if (k + 1 < ntiles) put(b ^ 1);
#pragma unroll
    for (int si = 0; si < NSI; ++si)
#pragma unroll
      for (int cb = 0; cb < NCB; ++cb) {
        cf[si][cb][0] = cn[si][cb][0];
        cf[si][cb][1] = cn[si][cb][1];
      }
#pragma unroll
    for (int jf = 0; jf < NJF; ++jf)
#pragma unroll
      for (int e = 0; e < NBS; ++e) bf[jf][e] = bn[jf][e];
    __syncthreads();
  }
  // lane holds rows 4 g + r of column m: d = d0 + 16 f + 4 g + r, j = h DH + NJF m + jf
  const int64_t DD = (int64_t)D * D;
  float* p = part + ((int64_t)z * 2 + (VAL ? 1 : 0)) * DD;
#pragma unroll
  for (int f = 0; f < 2; ++f)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int64_t o = (int64_t)(d0 + 16 * f + 4 * g + r) * D + h * DH + NJF * m;
      if constexpr (NJF == 4)
        *reinterpret_cast<float4*>(p + o) = make_float4(acc[f][0][r] * bscale, acc[f][1][r] * bscale,
                                                        acc[f][2][r] * bscale, acc[f][3][r] * bscale);
      else
        *reinterpret_cast<float2*>(p + o) = make_float2(acc[f][0][r] * bscale, acc[f][1][r] * bscale);
    }
}

// The B operands of both products as fragments, once per tile of 32 windows
// (every row group of the gradients reads the same ones): block (tile, kv),
// wave h.  Cp[tile][ks][cb][hi | lo][lane]: the first product's Cbd for k-step
// ks and column block cb (C = dS for the key, A for the value; lane (g, m):
// k = 32 ks + 8 g + j, column m); Bp[tile][h][jf][hi, lo | hi][lane]: scale-free
// q as hi + lo, or bf(dO), at windows 8 g + j, column h DH + NJF m + jf.  Rows
// past N are read clamped (their coefficients are zero).
template <int T, int DH, int H>
__global__ __launch_bounds__(64 * H) void k_kv_pack(const float* __restrict__ dS, const float* __restrict__ Ac,
                                                    const float* __restrict__ q, const float* __restrict__ dO, int N,
                                                    uint4* __restrict__ Ck, uint4* __restrict__ Cv,
                                                    uint4* __restrict__ Bq, uint4* __restrict__ Bd) {
  constexpr int D = H * DH, NJF = DH / 16;
  constexpr int NKS = KVW_NT * T / 32, WPC = 16 / H, NCB = 32 / T / WPC;
  const int h = threadIdx.x >> 6, l = threadIdx.x & 63, g = l >> 4, m = l & 15;
  const int64_t tl = blockIdx.x;
  const int n0 = (int)tl * KVW_NT;
  const bool val = blockIdx.y != 0;
  const float* __restrict__ C = val ? Ac : dS;
  uint4* __restrict__ Cp = val ? Cv : Ck;
  for (int ks = h; ks < NKS; ks += H)
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) {
      // lane's k = 32 ks + 8 g + j (window k / T, token k % T); column m:
      // window 32 ks / T + cb WPC + m / H, head m % H
      const int wcol = 32 * ks / T + cb * WPC + m / H, hh = m % H;
      float v[8];
#pragma unroll
      for (int jq = 0; jq < 2; ++jq) {
        const int k4 = 32 * ks + 8 * g + 4 * jq, w = k4 / T, t0 = k4 % T;
        const float4 c = *reinterpret_cast<const float4*>(C + ((uint32_t)min(n0 + w, N - 1) * H + hh) * T + t0);
        const bool on = w == wcol && n0 + w < N;
        v[4 * jq] = on ? c.x : 0.f;
        v[4 * jq + 1] = on ? c.y : 0.f;
        v[4 * jq + 2] = on ? c.z : 0.f;
        v[4 * jq + 3] = on ? c.w : 0.f;
      }
      uint4 hi, lo;
      kvw_split8(v, hi, lo);
      Cp[(((tl * NKS + ks) * NCB + cb) * 2) * 64 + l] = hi;
      Cp[(((tl * NKS + ks) * NCB + cb) * 2 + 1) * 64 + l] = lo;
    }
  float bv[8][NJF];
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const uint32_t o = (uint32_t)min(n0 + 8 * g + j, N - 1) * D + h * DH + NJF * m;
    const float* V = val ? dO : q;
    if constexpr (NJF == 4) {
      const float4 a = *reinterpret_cast<const float4*>(V + o);
      bv[j][0] = a.x; bv[j][1] = a.y; bv[j][2] = a.z; bv[j][3] = a.w;
    } else {
      const float2 a = *reinterpret_cast<const float2*>(V + o);
      bv[j][0] = a.x; bv[j][1] = a.y;
    }
  }
#pragma unroll
  for (int jf = 0; jf < NJF; ++jf) {
    float v[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) v[j] = bv[j][jf];
    uint4 hi, lo;
    kvw_split8(v, hi, lo);
    if (val) {
      Bd[((tl * H + h) * NJF + jf) * 64 + l] = hi;
    } else {
      Bq[(((tl * H + h) * NJF + jf) * 2) * 64 + l] = hi;
      Bq[(((tl * H + h) * NJF + jf) * 2 + 1) * 64 + l] = lo;
    }
  }
}

template <int T, int DH, int H>
__global__ __launch_bounds__(64 * H) void k_kv_wgrad(const uint16_t* __restrict__ X, const uint8_t* __restrict__ win,
                                                     const uint16_t* __restrict__ E, int e, int g,
                                                     const uint4* __restrict__ Ck, const uint4* __restrict__ Cv,
                                                     const uint4* __restrict__ Bq, const uint4* __restrict__ Bd, int N,
                                                     int nps, float scale, float* __restrict__ part) {
  __shared__ __align__(16) KvwLds<T, H> sm;
  // blocks are dealt to the 8 XCDs in turn (block L on XCD L % 8): logical
  // block lam = (L % 8) per + L / 8 gives each XCD a contiguous run of them,
  // i.e. whole window ranges (their D / 32 row groups, key then value), so
  // the ranges' rows of X and their fragments are fetched into that XCD's L2 once
  constexpr int ND = H * DH / KVW_DC;
  const int tot = (int)gridDim.x, per = tot / 8, L = (int)blockIdx.x;
  const int lam = L < 8 * per ? (L % 8) * per + L / 8 : L;
  const int x = lam % ND, kv = (lam / ND) & 1, z = lam / (2 * ND), S = tot / (2 * ND);
  if (kv == 0)
    kv_wgrad_body<T, DH, H, false>(sm, X, win, E, e, g, Ck, Bq, N, nps, scale, part, x * KVW_DC, z, S);
  else
    kv_wgrad_body<T, DH, H, true>(sm, X, win, E, e, g, Cv, Bd, N, nps, 1.f, part, x * KVW_DC, z, S);
}

// windows per range (a multiple of the tile) and number of ranges: about 256
// blocks of D / 32 row groups
static void kv_wgrad_split(int64_t N, int D, int& nps, int& S) {
  const int64_t tiles = (N + KVW_NT - 1) / KVW_NT;
  const int64_t want = std::max<int64_t>(1, std::min<int64_t>(tiles, (256 + D / KVW_DC - 1) / (D / KVW_DC)));
  nps = (int)((tiles + want - 1) / want) * KVW_NT;
  S = (int)((N + nps - 1) / nps);
}

// workspace: partial sums [S][2][D][D], then (16-byte units) Ck, Cv
// [tiles][T][2 H / T][2][64], Bq [tiles][D / 16][2][64], Bd [tiles][D / 16][64]
// (sized with the bound of the number of ranges, min(tiles, 256 / (D / 32)),
// which grows with N, so that a workspace sized for N windows serves every
// smaller batch; the number itself does not always grow with N)
int64_t kv_wgrad_ws_floats(int64_t N, int T, int D, int H) {
  if (N <= 0) return 0;
  const int64_t tiles = (N + KVW_NT - 1) / KVW_NT;
  const int64_t smax = std::max<int64_t>(1, std::min<int64_t>(tiles, (256 + D / KVW_DC - 1) / (D / KVW_DC)));
  return (int64_t)2 * smax * D * D + 4 * tiles * 64 * (2 * (int64_t)2 * H * 2 + (int64_t)D / 16 * 3);
}

// (the first product's column blocks need 32 / T windows per k-step to cover
// at least 16 / H windows: 2 H >= T)
bool kv_wgrad_built(int T, int D, int H) { return dx_rank1_built(T, D, H) && H <= 8 && 2 * H >= T; }

bool kv_wgrad_ready(int64_t N, int T, int D, int H, int e, int64_t ws_cap) {
  // 32-bit element offsets in the kernels; the gathered form needs e a multiple of 8
  return N > 0 && N * D < ((int64_t)1 << 29) && N * T * D < ((int64_t)1 << 30) && kv_wgrad_built(T, D, H) &&
         kv_wgrad_ws_floats(N, T, D, H) <= ws_cap && e % 8 == 0;
}

bool launch_kv_wgrad(const uint16_t* X, const uint8_t* win, const uint16_t* E, int e, int g, const float* dS,
                     const float* A, const float* q, const float* dO, int64_t N, int T, int D, int H, float scale,
                     float* ws, int64_t ws_cap, float* dWk, float* dWv, hipStream_t s) {
  if (!kv_wgrad_ready(N, T, D, H, win ? e : 8, ws_cap) || (!win && !X)) return false;
  if (dWv != dWk + (int64_t)D * D) return false;  // one split-K pass for both
  if (((uintptr_t)X | (uintptr_t)E | (uintptr_t)dS | (uintptr_t)A | (uintptr_t)q | (uintptr_t)dO | (uintptr_t)ws) & 15)
    return false;
  int nps, S;
  kv_wgrad_split(N, D, nps, S);
  const int DH = D / H;
  const int64_t tiles = (N + KVW_NT - 1) / KVW_NT;
  uint4* Ck = reinterpret_cast<uint4*>(ws + (int64_t)2 * S * D * D);
  uint4* Cv = Ck + tiles * 2 * H * 2 * 64;
  uint4* Bq = Cv + tiles * 2 * H * 2 * 64;
  uint4* Bd = Bq + tiles * (D / 16) * 2 * 64;
  const dim3 grid((unsigned)(2 * S * (D / KVW_DC)));
#define TRACE_KVW(T_, DH_, H_)                                                                                  \
  if (T == T_ && DH == DH_ && H == H_) {                                                                        \
    hipLaunchKernelGGL((k_kv_pack<T_, DH_, H_>), dim3((unsigned)tiles, 2), dim3(64 * H_), 0, s, dS, A, q, dO,   \
                       (int)N, Ck, Cv, Bq, Bd);                                                                 \
    hipLaunchKernelGGL((k_kv_wgrad<T_, DH_, H_>), grid, dim3(64 * H_), 0, s, X, win, E, e, g, Ck, Cv, Bq, Bd,   \
                       (int)N, nps, scale, ws);                                                                 \
  }
  TRACE_KVW(4, 32, 4) TRACE_KVW(8, 32, 4) TRACE_KVW(4, 64, 2)
  TRACE_KVW(4, 32, 8) TRACE_KVW(8, 32, 8) TRACE_KVW(4, 64, 4) TRACE_KVW(8, 64, 4)
  TRACE_KVW(4, 64, 8) TRACE_KVW(8, 64, 8)
#undef TRACE_KVW
  // the two gradients as one [2 D][D] product
  launch_splitk_reduce(ws, S, 2 * D, D, dWk, D, 0.f, nullptr, s);
  return true;
}

// dP[t][c] = sum_j sK[t][j] Wk[c][j] + sV[t][j] Wv[c][j], plus, for t = T-1,
// sQ[j] Wq[c][j] + sY[c]: the positional table's gradient sum_n dX[n][t], with
// the sums over windows taken before the products (weights as the operand
// copies: rounded to bf16 in bf16 models).  One wave per output, the lanes
// across j, the lane sums in a fixed tree.
__global__ __launch_bounds__(256) void k_pos_table_grad(const float* __restrict__ sKV, const float* __restrict__ sQ,
                                                        const float* __restrict__ sY, const float* __restrict__ Wq,
                                                        const float* __restrict__ Wk, const float* __restrict__ Wv,
                                                        int T, int D, int rb, float* __restrict__ dP) {
  const int i = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (i >= T * D) return;
  const int t = i / D, c = i % D;
  auto w = [&](const float* W, int j) { return rb ? round_bf(W[(int64_t)c * D + j]) : W[(int64_t)c * D + j]; };
  float acc = 0.f;
  for (int j = lane; j < D; j += 64) {
    acc = fmaf(sKV[t * D + j], w(Wk, j), acc);
    acc = fmaf(sKV[(T + t) * D + j], w(Wv, j), acc);
    if (t == T - 1) acc = fmaf(sQ[j], w(Wq, j), acc);
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) acc += __shfl_xor(acc, off, 64);
  if (lane == 0) dP[i] = t == T - 1 ? acc + sY[c] : acc;
}
// The same sums with one wave per weight row c for all T tokens: the block
// stages the window sums (2 T + 1 rows of D floats) in LDS, each wave reads its
// row's weights once (all of a lane's loads first), and each output's terms are
// added in the same order as above (bitwise the same results).
constexpr int PTG_ROWS = 8;  // weight rows (waves) per block
template <int T>
__global__ __launch_bounds__(64 * PTG_ROWS) void k_pos_table_grad_rows(const float* __restrict__ sKV,
                                                                       const float* __restrict__ sQ,
                                                                       const float* __restrict__ sY,
                                                                       const float* __restrict__ Wq,
                                                                       const float* __restrict__ Wk,
                                                                       const float* __restrict__ Wv, int D, int rb,
                                                                       float* __restrict__ dP) {
  constexpr int JMAX = 8;  // D <= 512
  __shared__ __align__(16) float S[(2 * T + 1) * 64 * JMAX];
  const int c = blockIdx.x * PTG_ROWS + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  const int nj = D / 64;  // D a multiple of 64
  const int cc = min(c, D - 1);  // (rows past D: loads clamped, nothing stored)
  float wk[JMAX], wv[JMAX], wq[JMAX];
#pragma unroll
  for (int i = 0; i < JMAX; ++i) {
    const int j = lane + 64 * min(i, nj - 1);  // (clamped; i < nj used)
    wk[i] = Wk[(int64_t)cc * D + j];
    wv[i] = Wv[(int64_t)cc * D + j];
    wq[i] = Wq[(int64_t)cc * D + j];
  }
  {  // every load of the staging first (float4; 2 T D + D is a multiple of 4)
    constexpr int NU = ((2 * T + 1) * 64 * JMAX / 4 + 64 * PTG_ROWS - 1) / (64 * PTG_ROWS);
    const int n4 = (2 * T * D) / 4, q4 = D / 4;
    float4 x[NU];
#pragma unroll
    for (int u = 0; u < NU; ++u) {
      const int i = threadIdx.x + 64 * PTG_ROWS * u;
      x[u] = i < n4 ? reinterpret_cast<const float4*>(sKV)[i]
                    : (i < n4 + q4 ? reinterpret_cast<const float4*>(sQ)[i - n4] : make_float4(0.f, 0.f, 0.f, 0.f));
    }
#pragma unroll
    for (int u = 0; u < NU; ++u) {
      const int i = threadIdx.x + 64 * PTG_ROWS * u;
      if (i < n4 + q4) reinterpret_cast<float4*>(S)[i] = x[u];
    }
  }
  __syncthreads();
  if (c >= D) return;
  if (rb) {
#pragma unroll
    for (int i = 0; i < JMAX; ++i) {
      wk[i] = round_bf(wk[i]);
      wv[i] = round_bf(wv[i]);
      wq[i] = round_bf(wq[i]);
    }
  }
  float acc[T];
#pragma unroll
  for (int t = 0; t < T; ++t) acc[t] = 0.f;
#pragma unroll
  for (int i = 0; i < JMAX; ++i) {
    if (i < nj) {
      const int j = lane + 64 * i;
#pragma unroll
      for (int t = 0; t < T; ++t) {
        acc[t] = fmaf(S[t * D + j], wk[i], acc[t]);
        acc[t] = fmaf(S[(T + t) * D + j], wv[i], acc[t]);
        if (t == T - 1) acc[t] = fmaf(S[2 * T * D + j], wq[i], acc[t]);
      }
    }
  }
#pragma unroll
  for (int t = 0; t < T; ++t) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) acc[t] += __shfl_xor(acc[t], off, 64);
  }
  if (lane == 0) {
#pragma unroll
    for (int t = 0; t < T; ++t) dP[t * D + c] = t == T - 1 ? acc[t] + sY[c] : acc[t];
  }
}

void launch_pos_table_grad(const float* sKV, const float* sQ, const float* sY, const float* Wq, const float* Wk,
                           const float* Wv, int T, int D, int rb, float* dP, hipStream_t s) {
  if (D % 64 == 0 && D <= 512 && (T == 4 || T == 8) && ((uintptr_t)sKV & 15) == 0 && ((uintptr_t)sQ & 15) == 0) {
    const dim3 grid((unsigned)((D + PTG_ROWS - 1) / PTG_ROWS));
    if (T == 8)
      hipLaunchKernelGGL(k_pos_table_grad_rows<8>, grid, dim3(64 * PTG_ROWS), 0, s, sKV, sQ, sY, Wq, Wk, Wv, D, rb,
                         dP);
    else
      hipLaunchKernelGGL(k_pos_table_grad_rows<4>, grid, dim3(64 * PTG_ROWS), 0, s, sKV, sQ, sY, Wq, Wk, Wv, D, rb,
                         dP);
    return;
  }
  hipLaunchKernelGGL(k_pos_table_grad, dim3((unsigned)((T * D + 3) / 4)), dim3(256), 0, s, sKV, sQ, sY, Wq, Wk, Wv,
                     T, D, rb, dP);
}

// ------------------------------------------------------ embedding backward ----
// dE[v][c] = sum over positions q = n*W + p with win[q] == v of dX[q*e + c]
// (the W token slots of a window are W consecutive e-vectors of dX, D = g*e,
// so position q reads row q of dX viewed as [N*W][e]).
// Deterministic, with dX read once: the positions are counting-sorted by byte
// value, stably (k_emb_hist, k_emb_colscan, k_emb_pieces, k_emb_scatter); each
// byte's sorted run is cut into pieces of EMB_PIECE positions, each summed in
// order by one wave (k_emb_piece); the pieces of a byte are added in a fixed
// order (k_emb_sum).
// The order of every sum depends on the input bytes alone.
constexpr int EMB_CS = 2048;    // positions per block of the counting sort
constexpr int EMB_PIECE = 256;  // positions per piece

struct EmbWs {
  int *cnt, *off, *tot, *base, *pstart, *piece, *perm;
  float* part;
};
static EmbWs emb_ws(float* ws, int64_t M, int e) {
  const int64_t nb = (M + EMB_CS - 1) / EMB_CS, pmax = (M + EMB_PIECE - 1) / EMB_PIECE + 256;
  EmbWs w;
  w.cnt = (int*)ws;
  w.off = w.cnt + nb * 256;
  w.tot = w.off + nb * 256;
  w.base = w.tot + 256;
  w.pstart = w.base + 256;
  w.piece = w.pstart + 260;
  w.perm = w.piece + 3 * pmax;
  // the piece sums start 16-byte aligned (if ws is)
  w.part = ws + ((w.perm + M - (int*)ws + 3) & ~(int64_t)3);
  (void)e;
  return w;
}
int64_t embed_bwd_ws_floats(int64_t M, int e) {
  const int64_t nb = (M + EMB_CS - 1) / EMB_CS, pmax = (M + EMB_PIECE - 1) / EMB_PIECE + 256;
  return 2 * nb * 256 + 512 + 260 + 3 * pmax + M + 3 + pmax * e;
}

// cnt[b][v] = number of positions of block b (EMB_CS positions) holding byte v
// (integer counts: the order of the LDS atomic adds does not matter)
__global__ __launch_bounds__(1024) void k_emb_hist(const uint8_t* __restrict__ win, int M, int* __restrict__ cnt) {
  __shared__ int h[256];
  if (threadIdx.x < 256) h[threadIdx.x] = 0;
  __syncthreads();
  const int q0 = blockIdx.x * EMB_CS;
  for (int u = threadIdx.x; u < EMB_CS; u += 1024) {
    const int q = q0 + u;
    if (q < M) atomicAdd(&h[win[q]], 1);
  }
  __syncthreads();
  if (threadIdx.x < 256) cnt[blockIdx.x * 256 + threadIdx.x] = h[threadIdx.x];
}

// Workgroup v: off[b][v] = number of v in blocks before b, tot[v] = all of them
// (thread t takes a contiguous range of blocks; exclusive scan over threads).
__global__ __launch_bounds__(256) void k_emb_colscan(const int* __restrict__ cnt, int nb, int* __restrict__ off,
                                                     int* __restrict__ tot) {
  __shared__ int sc[256];
  const int v = blockIdx.x, t = threadIdx.x;
  const int per = (nb + 255) / 256, b0 = min(nb, t * per), b1 = min(nb, b0 + per);
  int s = 0;
  for (int b = b0; b < b1; ++b) s += cnt[b * 256 + v];
  sc[t] = s;
  __syncthreads();
  for (int d = 1; d < 256; d <<= 1) {
    const int a = t >= d ? sc[t - d] : 0;
    __syncthreads();
    sc[t] += a;
    __syncthreads();
  }
  int run = sc[t] - s;
  for (int b = b0; b < b1; ++b) {
    off[b * 256 + v] = run;
    run += cnt[b * 256 + v];
  }
  if (t == 255) tot[v] = sc[255];
}

// One workgroup: base[v] = sorted position of the first v (counts of smaller
// bytes); byte v's run is cut into pieces (v, first sorted position, length),
// numbered from pstart[v]; pstart[256] = number of pieces.
__global__ __launch_bounds__(1024) void k_emb_pieces(const int* __restrict__ tot, int* __restrict__ base,
                                                     int* __restrict__ pstart, int* __restrict__ piece) {
  __shared__ int tb[256], np[256], ps[257];
  const int t = threadIdx.x;
  int total = 0, npv = 0;
  if (t < 256) {
    total = tot[t];
    npv = (total + EMB_PIECE - 1) / EMB_PIECE;
    tb[t] = total;
    np[t] = npv;
  }
  __syncthreads();
  for (int d = 1; d < 256; d <<= 1) {
    int a = 0, c = 0;
    if (t < 256 && t >= d) {
      a = tb[t - d];
      c = np[t - d];
    }
    __syncthreads();
    if (t < 256) {
      tb[t] += a;
      np[t] += c;
    }
    __syncthreads();
  }
  if (t < 256) {
    base[t] = tb[t] - total;
    ps[t] = np[t] - npv;
    pstart[t] = np[t] - npv;
  }
  if (t == 0) {
    ps[256] = np[255];
    pstart[256] = np[255];
  }
  __syncthreads();
  // piece j: its byte by binary search over ps
  for (int j = t; j < ps[256]; j += 1024) {
    int lo = 0, hi = 256;  // ps[lo] <= j < ps[hi]
    while (hi - lo > 1) {
      const int mid = (lo + hi) >> 1;
      if (ps[mid] <= j)
        lo = mid;
      else
        hi = mid;
    }
    const int k = j - ps[lo], bv = tb[lo] - (lo > 0 ? tb[lo - 1] : 0);
    piece[3 * j] = lo;
    piece[3 * j + 1] = (tb[lo] - bv) + k * EMB_PIECE;
    piece[3 * j + 2] = min(EMB_PIECE, bv - k * EMB_PIECE);
  }
}

// perm[sorted position] = position, stable: block b places its positions in
// increasing order, 1024 per round; within a wave the rank among lanes with the
// same byte comes from ballots on the byte's 8 bits, across the round's waves
// from their counts in wave order.
__global__ __launch_bounds__(1024) void k_emb_scatter(const uint8_t* __restrict__ win, int M,
                                                      const int* __restrict__ off, const int* __restrict__ base,
                                                      int* __restrict__ perm) {
  __shared__ int run[256];
  __shared__ int wc[16][256];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  if (tid < 256) run[tid] = base[tid] + off[blockIdx.x * 256 + tid];
  const int q0 = blockIdx.x * EMB_CS;
  const uint64_t below = lane == 0 ? 0ull : (~0ull >> (64 - lane));
  constexpr int R = EMB_CS / 1024;
  int vr[R];
#pragma unroll
  for (int r = 0; r < R; ++r) vr[r] = win[min(q0 + r * 1024 + tid, M - 1)];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    for (int i = tid; i < 16 * 256; i += 1024) (&wc[0][0])[i] = 0;
    __syncthreads();
    const int q = q0 + r * 1024 + tid;
    const bool live = q < M;
    const int v = live ? vr[r] : 0;
    uint64_t same = __ballot(live);
#pragma unroll
    for (int bit = 0; bit < 8; ++bit) {
      const uint64_t bb = __ballot((v >> bit) & 1);
      same &= ((v >> bit) & 1) ? bb : ~bb;
    }
    const int rank = __popcll(same & below);
    if (live && rank == 0) wc[wv][v] = __popcll(same);
    __syncthreads();
    if (live) {
      int pos = run[v] + rank;
      for (int w2 = 0; w2 < wv; ++w2) pos += wc[w2][v];
      perm[pos] = q;
    }
    __syncthreads();
    if (tid < 256) {
      int t = 0;
#pragma unroll
      for (int w2 = 0; w2 < 16; ++w2) t += wc[w2][tid];
      run[tid] += t;
    }
    __syncthreads();
  }
}

// part[p][c] = sum of the dX rows of piece p's positions in sorted order, one
// wave per piece.  e <= 64 dividing 64: lane l takes feature l % e of the
// positions u with u % (64 / e) == l / e, and the 64 / e partial sums are added
// at the end in a fixed tree; other e: lanes c and c + 64 take features c and
// c + 64 of every position (e <= 128).
__global__ __launch_bounds__(64) void k_emb_piece(const float* __restrict__ dX, int e, const int* __restrict__ perm,
                                                  const int* __restrict__ piece, const int* __restrict__ pstart,
                                                  float* __restrict__ part) {
  constexpr int B = 32;  // loads in flight per lane
  const int p = blockIdx.x;
  if (p >= pstart[256]) return;
  const int st = piece[3 * p + 1], len = piece[3 * p + 2];
  const int lane = threadIdx.x;
  const int ipl = (e <= 64 && 64 % e == 0) ? 64 / e : 1;  // positions per load instruction
  const int sub = ipl > 1 ? lane / e : 0;
  // every load is made, from a clamped feature; lanes past the features add nothing
  const int f0 = ipl > 1 ? lane - sub * e : min(lane, e - 1), f1 = min(lane + 64, e - 1);
  float a0 = 0.f, a1 = 0.f;
  for (int i0 = 0; i0 < len; i0 += 64) {
    const int n = min(64, len - i0);
    const int my = perm[st + i0 + min(lane, n - 1)];
    for (int u0 = 0; u0 < n; u0 += B * ipl) {
      float x0[B], x1[B];
#pragma unroll
      for (int u = 0; u < B; ++u) {
        // this lane's position: u0 + u * ipl + sub (clamped; masked below)
        const int j = u0 + u * ipl + sub;
        const int q = ipl > 1 ? __builtin_amdgcn_ds_bpermute(4 * min(j, n - 1), my)
                              : __builtin_amdgcn_readlane(my, min(u0 + u, n - 1));
        x0[u] = dX[(int64_t)q * e + f0];
        if (e > 64) x1[u] = dX[(int64_t)q * e + f1];
      }
#pragma unroll
      for (int u = 0; u < B; ++u) {
        if (u0 + u * ipl + sub < n) {
          a0 += x0[u];
          if (e > 64) a1 += x1[u];
        }
      }
    }
  }
  // partial sums of the position classes, added in a fixed tree
  for (int d = 1; d < ipl; d <<= 1) a0 += __shfl_down(a0, d * e, 64);
  if (lane < e) part[(int64_t)p * e + lane] = a0;
  if (e > 64 && lane + 64 < e) part[(int64_t)p * e + lane + 64] = a1;
}

// dE[v][c] = sum of byte v's pieces: row group rg of 256 / e takes every
// (256 / e)-th piece in order, then the groups are added in order
__global__ __launch_bounds__(256) void k_emb_sum(const float* __restrict__ part, const int* __restrict__ pstart, int e,
                                                 float* __restrict__ dE) {
  __shared__ float red[256];
  const int v = blockIdx.x, tid = threadIdx.x;
  const int RG = 256 / e, rg = tid / e, c = tid - rg * e;
  const int p0 = pstart[v], p1 = pstart[v + 1];
  float s = 0.f;
  if (rg < RG) {
#pragma unroll 4
    for (int p = p0 + rg; p < p1; p += RG) s += part[(int64_t)p * e + c];
  }
  red[tid] = s;
  __syncthreads();
  if (tid < e) {
    float t = 0.f;
    for (int q = 0; q < RG; ++q) t += red[q * e + tid];
    dE[v * e + tid] = t;
  }
}

void launch_embed_bwd(const uint8_t* win, const float* dX, int64_t N, int W, int e, float* dE, float* ws,
                      hipStream_t s) {
  const int64_t M = N * W;
  if (M <= 0) {
    launch_zero(dE, (int64_t)256 * e, s);
    return;
  }
  const EmbWs w = emb_ws(ws, M, e);
  const int nb = (int)((M + EMB_CS - 1) / EMB_CS);
  const int pmax = (int)((M + EMB_PIECE - 1) / EMB_PIECE + 256);
  hipLaunchKernelGGL(k_emb_hist, dim3(nb), dim3(1024), 0, s, win, (int)M, w.cnt);
  hipLaunchKernelGGL(k_emb_colscan, dim3(256), dim3(256), 0, s, (const int*)w.cnt, nb, w.off, w.tot);
  hipLaunchKernelGGL(k_emb_pieces, dim3(1), dim3(1024), 0, s, (const int*)w.tot, w.base, w.pstart, w.piece);
  hipLaunchKernelGGL(k_emb_scatter, dim3(nb), dim3(1024), 0, s, win, (int)M, (const int*)w.off,
                     (const int*)w.base, w.perm);
  hipLaunchKernelGGL(k_emb_piece, dim3(pmax), dim3(64), 0, s, dX, e, (const int*)w.perm, (const int*)w.piece,
                     (const int*)w.pstart, w.part);
  hipLaunchKernelGGL(k_emb_sum, dim3(256), dim3(256), 0, s, (const float*)w.part, (const int*)w.pstart, e, dE);
}

// byte-embedding part of the kept tokens: G[n][t][c] = E[byte][c % e] (the
// operand value).  The token is X = G + P[t]; the weight gradients X^T.dZ are
// formed as G^T.dZ (a GEMM) plus P^T.(sum over windows of dZ) (k_pos_grad).
template <bool BF>
__global__ __launch_bounds__(256) void k_gather_kept(const uint8_t* __restrict__ win, int64_t rows,
                                                     const typename Mma<BF>::T* __restrict__ E, int T, int D, int e,
                                                     int g, void* __restrict__ X) {
  // thread: four consecutive columns of one token row (row = n*T + t); e is a
  // multiple of 4, so the four share one byte.  BF: X holds the bf16 operand
  // values themselves; otherwise fp32
  typedef Mma<BF> M;
  const uint32_t q4 = (uint32_t)D / 4;
  const uint32_t i = blockIdx.x * 256u + threadIdx.x;  // the grid has fewer than 2^32 threads
  if ((int64_t)i >= rows * q4) return;
  const uint32_t row32 = i / q4;
  const int64_t row = row32;
  const int c = (int)(i - row32 * q4) * 4;
  const int j = c / e, cc = c - j * e;
  // the byte of token t, group slot j of window n sits at win[n*T*g + t*g + j] = win[row*g + j]
  const int byte = win[row * g + j];
  const typename M::T* src = E + byte * e + cc;
  if constexpr (BF)
    *reinterpret_cast<uint2*>((uint16_t*)X + row * D + c) =
        make_uint2((uint32_t)src[0] | ((uint32_t)src[1] << 16), (uint32_t)src[2] | ((uint32_t)src[3] << 16));
  else
    *reinterpret_cast<float4*>((float*)X + row * D + c) =
        make_float4(M::val(src[0]), M::val(src[1]), M::val(src[2]), M::val(src[3]));
}
// bf16 with e a multiple of 8: units of eight consecutive columns, one 16-byte
// load of the embedding row and one 16-byte store each.  A block takes
// GK_U * 256 consecutive units, a thread GK_U of them 256 apart, all byte loads
// first, then all row loads, then the stores.
constexpr int GK_U = 4;
__global__ __launch_bounds__(256) void k_gather_kept8(const uint8_t* __restrict__ win, int64_t rows, int wstride,
                                                      const uint16_t* __restrict__ E, int D, int e,
                                                      uint16_t* __restrict__ X) {
  const uint32_t q8 = (uint32_t)D / 8;
  const uint32_t nu = (uint32_t)rows * q8;  // the grid has fewer than 2^32 units
  const uint32_t i0 = blockIdx.x * (256u * GK_U) + threadIdx.x;
  int byte[GK_U], cc[GK_U];
#pragma unroll
  for (int u = 0; u < GK_U; ++u) {
    const uint32_t i = min(i0 + 256u * u, nu - 1);  // clamped; stored only inside
    const uint32_t row = i / q8;
    const int c = (int)(i - row * q8) * 8;
    const int j = c / e;
    cc[u] = c - j * e;
    byte[u] = win[(int64_t)row * wstride + j];
  }
  typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;
  u32x4 v[GK_U];
#pragma unroll
  for (int u = 0; u < GK_U; ++u) {
    const uint4 x = *reinterpret_cast<const uint4*>(E + byte[u] * e + cc[u]);
    v[u] = u32x4{x.x, x.y, x.z, x.w};
  }
#pragma unroll
  for (int u = 0; u < GK_U; ++u) {
    const uint32_t i = i0 + 256u * u;
    if (i < nu) __builtin_nontemporal_store(v[u], reinterpret_cast<u32x4*>(X + (int64_t)i * 8));
  }
}
void launch_gather_kept(bool bf, const uint8_t* win, int64_t N, const void* E, int T, int D, int e, int g, void* X,
                        hipStream_t s) {
  const int64_t rows = N * T;
  if (rows <= 0) return;
  if (bf && e % 8 == 0 && ((uintptr_t)E & 15) == 0 && ((uintptr_t)X & 15) == 0 &&
      rows * (D / 8) < ((int64_t)1 << 31)) {
    const dim3 grid8((unsigned)((rows * (D / 8) + 256 * GK_U - 1) / (256 * GK_U)));
    hipLaunchKernelGGL(k_gather_kept8, grid8, dim3(256), 0, s, win, rows, g, (const uint16_t*)E, D, e,
                       (uint16_t*)X);
    return;
  }
  const dim3 grid((unsigned)((rows * (D / 4) + 255) / 256));
  if (bf)
    hipLaunchKernelGGL(k_gather_kept<true>, grid, dim3(256), 0, s, win, rows, (const uint16_t*)E, T, D, e, g, X);
  else
    hipLaunchKernelGGL(k_gather_kept<false>, grid, dim3(256), 0, s, win, rows, (const float*)E, T, D, e, g, X);
}

bool launch_gather_last(const uint8_t* win, int64_t N, const uint16_t* E, int T, int D, int e, int g, uint16_t* X,
                        hipStream_t s) {
  if (N <= 0) return true;
  if (e % 8 != 0 || ((uintptr_t)E & 15) != 0 || ((uintptr_t)X & 15) != 0 || N * (D / 8) >= ((int64_t)1 << 31))
    return false;
  // the last token's group of window n starts (T - 1) g bytes into its W = T g bytes
  const dim3 grid8((unsigned)((N * (D / 8) + 256 * GK_U - 1) / (256 * GK_U)));
  hipLaunchKernelGGL(k_gather_kept8, grid8, dim3(256), 0, s, win + (int64_t)(T - 1) * g, N, T * g, E, D, e, X);
  return true;
}

// Positional part of a projection's weight gradient:
// dW[i][j] += sum_{u < nt} P[t0 + u][i] * S[u][j], with S[u] = sum over windows
// of dZ at token t0 + u (column sums, formed beforehand in a fixed order); the
// sum over u runs in increasing order.
template <bool BF>
__global__ void k_pos_grad(const typename Mma<BF>::T* __restrict__ P, const float* __restrict__ S, int t0, int nt,
                           int D, float* __restrict__ dW) {
  typedef Mma<BF> M;
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= (int64_t)D * D) return;
  const int r = (int)(i / D), c = (int)(i % D);
  float acc = 0.f;
  for (int u = 0; u < nt; ++u) acc += M::val(P[(t0 + u) * D + r]) * S[u * D + c];
  dW[i] += acc;
}
void launch_pos_grad(bool bf, const void* P, const float* S, int t0, int nt, int D, float* dW, hipStream_t s) {
  const dim3 grid((unsigned)(((int64_t)D * D + 255) / 256));
  if (bf)
    hipLaunchKernelGGL(k_pos_grad<true>, grid, dim3(256), 0, s, (const uint16_t*)P, S, t0, nt, D, dW);
  else
    hipLaunchKernelGGL(k_pos_grad<false>, grid, dim3(256), 0, s, (const float*)P, S, t0, nt, D, dW);
}

// Up to three positional parts in one launch (blockIdx.y = the job), each as
// k_pos_grad computes it.
struct PosGradJobs {
  const float* S[3];
  float* dW[3];
  int t0[3], nt[3];
};
template <bool BF>
__global__ void k_pos_grad3(const typename Mma<BF>::T* __restrict__ P, PosGradJobs jb, int D) {
  typedef Mma<BF> M;
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= (int64_t)D * D) return;
  const int y = blockIdx.y;
  // the job's fields, selected with constant indexes (blockIdx.y is uniform)
  const float* S = y == 0 ? jb.S[0] : (y == 1 ? jb.S[1] : jb.S[2]);
  float* dW = y == 0 ? jb.dW[0] : (y == 1 ? jb.dW[1] : jb.dW[2]);
  const int t0 = y == 0 ? jb.t0[0] : (y == 1 ? jb.t0[1] : jb.t0[2]);
  const int nt = y == 0 ? jb.nt[0] : (y == 1 ? jb.nt[1] : jb.nt[2]);
  const int r = (int)(i / D), c = (int)(i % D);
  float acc = 0.f;
  for (int u = 0; u < nt; ++u) acc += M::val(P[(t0 + u) * D + r]) * S[u * D + c];
  dW[i] += acc;
}
void launch_pos_grad3(bool bf, const void* P, const float* const* S, const int* t0, const int* nt, float* const* dW,
                      int njobs, int D, hipStream_t s) {
  if (njobs < 1 || njobs > 3) return;
  PosGradJobs jb{};
  for (int j = 0; j < njobs; ++j) {
    jb.S[j] = S[j];
    jb.dW[j] = dW[j];
    jb.t0[j] = t0[j];
    jb.nt[j] = nt[j];
  }
  const dim3 grid((unsigned)(((int64_t)D * D + 255) / 256), (unsigned)njobs);
  if (bf)
    hipLaunchKernelGGL(k_pos_grad3<true>, grid, dim3(256), 0, s, (const uint16_t*)P, jb, D);
  else
    hipLaunchKernelGGL(k_pos_grad3<false>, grid, dim3(256), 0, s, (const float*)P, jb, D);
}

// -------------------------------------------------------------------- Adam ----
// Kingma & Ba, Alg. 1, with the bias corrections bc1 = 1 - beta1^t and
// bc2 = 1 - beta2^t supplied by the host.  Each product and sum is rounded on
// its own (contraction into fused multiply-adds is off), in the order m = b1*m + (1-b1)*g,
// v = b2*v + ((1-b2)*g)*g, theta -= (lr * m/bc1) / (sqrt(v/bc2) + eps).
__device__ __forceinline__ void adam1(float& th, float g, float& m, float& v, float lr, float b1, float b2, float eps,
                                      float bc1, float bc2) {
#pragma clang fp contract(off)
  const float omb1 = __fsub_rn(1.f, b1), omb2 = __fsub_rn(1.f, b2);
  const float mi = __fadd_rn(__fmul_rn(b1, m), __fmul_rn(omb1, g));
  const float vi = __fadd_rn(__fmul_rn(b2, v), __fmul_rn(__fmul_rn(omb2, g), g));
  m = mi;
  v = vi;
  const float mhat = __fdiv_rn(mi, bc1);
  const float vhat = __fdiv_rn(vi, bc2);
  // correctly rounded sqrt: the fp64 root rounded once to fp32 (53 >= 2*24 + 2
  // bits, so the two roundings give the singly rounded result)
  const float root = (float)__dsqrt_rn((double)vhat);
  const float step = __fdiv_rn(__fmul_rn(lr, mhat), __fadd_rn(root, eps));
  th = __fsub_rn(th, step);
}
// four parameters per thread with 16-byte loads and stores (n % 4 elements at
// the end one per thread)
__global__ void k_adam(float* __restrict__ theta, const float* __restrict__ grad, float* __restrict__ m,
                       float* __restrict__ v, int64_t n, float lr, float b1, float b2, float eps, float bc1,
                       float bc2) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t n4 = n / 4;
  if (i < n4) {
    float4 t = reinterpret_cast<float4*>(theta)[i];
    const float4 g = reinterpret_cast<const float4*>(grad)[i];
    float4 mm = reinterpret_cast<float4*>(m)[i];
    float4 vv = reinterpret_cast<float4*>(v)[i];
    adam1(t.x, g.x, mm.x, vv.x, lr, b1, b2, eps, bc1, bc2);
    adam1(t.y, g.y, mm.y, vv.y, lr, b1, b2, eps, bc1, bc2);
    adam1(t.z, g.z, mm.z, vv.z, lr, b1, b2, eps, bc1, bc2);
    adam1(t.w, g.w, mm.w, vv.w, lr, b1, b2, eps, bc1, bc2);
    reinterpret_cast<float4*>(theta)[i] = t;
    reinterpret_cast<float4*>(m)[i] = mm;
    reinterpret_cast<float4*>(v)[i] = vv;
  } else {
    const int64_t j = 4 * n4 + (i - n4);
    if (j < n) adam1(theta[j], grad[j], m[j], v[j], lr, b1, b2, eps, bc1, bc2);
  }
}
void launch_adam(float* theta, const float* grad, float* m, float* v, int64_t n, float lr, float b1, float b2,
                 float eps, float bc1, float bc2, hipStream_t s, hipEvent_t t0, hipEvent_t t1) {
  const int64_t threads = n / 4 + n % 4;
  // t0 / t1 (may be null) take the dispatch's own start and end time stamps
  hipExtLaunchKernelGGL(k_adam, dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, s, t0, t1, 0, theta, grad, m,
                        v, n, lr, b1, b2, eps, bc1, bc2);
}
