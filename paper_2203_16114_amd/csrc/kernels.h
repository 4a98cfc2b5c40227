// Launch interface between the C-ABI layer (api.cpp) and the HIP kernels.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

// Windows are addressed by a flat index n = b * n_steps + s over (stream, step);
// a launch covers n0 .. n0 + N - 1.  Window n reads bytes
// streams[b*stride + pos0 + s - W .. + W - 1] and targets streams[b*stride + pos0 + s].
struct WinArgs {
  const uint8_t* streams;
  int64_t stride, pos0;
  int32_t n_steps;
  int64_t n0, N;
};

struct AttnArgs {
  WinArgs w;
  const void* E;  // operand copy [256][e]
  const void* P;  // operand copy [T][D] (zeros when the positional table is off)
  const float* PW; // [3][T][D]: P.Wq, P.Wk, P.Wv (fp32), the positional parts of the projections
  int32_t e, g;
  const uint4 *Wq, *Wk, *Wv, *Wo;  // packed operand copies
  float* h0;                       // [N][D]: Attn + X, the residual stream entering the FFN
  float scale;                     // 1/sqrt(head width)
  float scale4;                    // (head width)^-1/4 (Performer)
  int32_t token_only;              // 1: the per-token kernel whatever the launch shape
  const float* Xin;                // later layers: input rows [N][T][D] (fp32; NULL: byte-group tokens)
  const uint4* Om;                 // Performer: packed random projection (NULL: softmax attention)
  int32_t nfeat;                   // Performer: features (a multiple of 16)
  // kept activations for the backward (all NULL unless kept), indexed by local window
  uint8_t* kwin;  // [N][W]
  float* kq;      // [N][D]     query of the last token
  float* kK;      // [N][T][D]
  float* kV;      // [N][T][D]
  float* kA;      // [N][H][T]  attention weights of the last row
  float* kO;      // [N][D]     attention output as the operand of Wo
};

struct FfnArgs {
  WinArgs w;
  const float* h0;                 // [N][D]
  const uint4 *W1, *W2, *Wout;     // packed operand copies
  const float* bout;               // [256]
  int32_t F, k;
  int64_t wstride;                 // uint4 between the packed W1 (W2) copies of two repeats; 0: shared
  float* bits;                     // [n0 + N] global window index
  float* logits;                   // nullable, [n0 + N][256]
  void* kY;                        // nullable, [k+1][N][D]: Y_0 .. Y_k as operand values (bf16 or fp32)
  float* kU;                       // nullable, [k][N][F]
  uint16_t* kG;                    // nullable, [k][N][F] bf16: GELU(U) as the operand values (bf16 path)
  float* kZ;                       // nullable, [N][256]
  int32_t* ktgt;                   // nullable, [N]
};

typedef void (*attn_fn)(const AttnArgs&, hipStream_t);
typedef void (*ffn_fn)(const FfnArgs&, hipStream_t);

// NULL when no kernel is built for the shape.
attn_fn find_attn(bool bf, int T, int D, int DH);
ffn_fn find_ffn(bool bf, int D);

void launch_zero(void* p, int64_t n32, hipStream_t s);
void launch_step_ce(const float* bits, int32_t n_streams, int32_t n_steps, double* out, hipStream_t s);
// One part of the operand refresh (all parts run in one launch):
//   RJ_CVT   dst[i] = operand(src[i]), i < K
//   RJ_PACK  fragment-packed operand copy of the [K][N] row-major src, each value times scale
//   RJ_PTAB  PW[w][t][j] = sum_i P[t][i] W_w[i][j] for w = q, k, v, t < K (= T: 4 or 8), j < N (= D: a multiple
//            of 64, at most 512), with the operand
//            values of P (src; zero if use_pos is 0) and of W_q (src2, W_k and W_v following it in the master)
//   RJ_ZERO  K 32-bit words of dst cleared
//   RJ_PACKT as RJ_PACK for the transpose of src: the copy of [K][N] src^T, src being [N][K] row-major
//   RJ_CVT8  as RJ_CVT, eight values per thread (K a multiple of 8, src and dst 16-byte aligned)
enum { RJ_CVT = 0, RJ_PACK = 1, RJ_PTAB = 2, RJ_ZERO = 3, RJ_PACKT = 4, RJ_CVT8 = 5 };
struct RefreshJob {
  const float* src;
  const float* src2;
  void* dst;
  int kind, K, N, use_pos;
  float scale;
};
constexpr int REFRESH_MAX_JOBS = 13;
// Runs jobs[0..n) on stream s; false (nothing launched) for an unsupported job.
bool launch_refresh(bool bf, const RefreshJob* jobs, int n, hipStream_t s);

// ---- backward building blocks (bwd.hip) ----
struct GemmArgs {
  int M, N, K;
  const float* A;
  int64_t sam, sak;  // A(m,k) = A[m*sam + k*sak]
  const float* B;
  int64_t sbk, sbn;  // B(k,n) = B[k*sbk + n*sbn]
  float* C;
  int64_t ldc;       // C(m,n) = C[m*ldc + n]
  int roundA, roundB;  // round that operand to bf16 (RNE) as it is read
  float beta;          // C = beta*Cin + A.B  (beta 0 or 1)
  // nullable: the addend of beta (laid out as C, ldc apart); NULL: C itself
  const float* Cin;
  // nullable: B formed from rank-one rows, B(k, n) = (r1c[(w H + n / dh) T + t] . V(w, n)) . r1scale
  // for k = w T + t, with V(w, n) = B[w*sbk + n] (sbn = 1; rounded to bf16 first if r1round) and
  // T = 2^r1tsh, dh = 2^r1dsh, H = r1H (the key and value gradients of the last query row);
  // fp32 B split into hi and lo, bf16 kernels only
  const float* r1c;
  int r1tsh, r1dsh, r1H, r1round;
  float r1scale;
  // nullable: C = (A.B) * GELU'(gelu_u) elementwise, gelu_u laid out as C
  // (the backward of the FFN activation fused into its product); needs beta 0
  const float* gelu_u;
  // that operand is stored as bf16 (A / B then point at bf16 elements and the
  // strides count them); only the bf16 kernel reads it, and it must be rounded
  int halfA, halfB;
  // C is written as bf16 (rounded to nearest even; C then points at bf16
  // elements); needs beta 0, and the product is not split over k
  int halfC;
};
// Deterministic: split-K partials are summed in a fixed order.  The split count
// depends only on (M, N, K, ws_cap); gemm_ws_floats(M, N, K) floats let it
// reach its preferred value.
int64_t gemm_ws_floats(int M, int N, int K);
// false only when an operand or result stored as bf16 does not fit the bf16 kernel
bool launch_gemm(const GemmArgs& g, float* ws, int64_t ws_cap, hipStream_t s);
// C = beta*C + A1.B1 + A2.B2: g and g2 share M, N, C, ldc, beta and rounding
// flags; one launch when the bf16 kernel takes both, else two
void launch_gemm2(const GemmArgs& g, const GemmArgs& g2, float* ws, int64_t ws_cap, hipStream_t s);
void launch_splitk_reduce(const float* ws, int splits, int M, int N, float* C, int64_t ldc, float beta,
                          const float* cin, hipStream_t s);
// bgemm.hip: false (nothing launched) when the product is not one it takes;
// g2 (nullable) is a second K segment summed into the same result
// force: 0 the kernel the shape calls for, 1 the 128-tile kernel, 2 the 256-tile kernel
bool launch_bgemm(const GemmArgs& g, const GemmArgs* g2, float* ws, int64_t ws_cap, hipStream_t s, int force = 0);
int64_t bgemm_ws_floats(int M, int N, int K);

void launch_colsum(const float* in, int64_t rows, int64_t cols, int64_t ld, float* out, float beta, float* ws,
                   hipStream_t s);
int64_t colsum_ws_floats(int64_t cols);
void launch_ce_grad(const float* z, const int32_t* tgt, int64_t N, float* dz, hipStream_t s);
void launch_gelu_fwd_round(const float* U, float* G, int64_t n, int round, hipStream_t s);
void launch_gelu_bwd(const float* dG, const float* U, float* dU, int64_t n, hipStream_t s);
// dS (nullable): [N][H][T] gradients of the attention scores of the last row
// dK, dV may be NULL (not written; their sums over windows still are)
void launch_attn_bwd(const float* dO, const float* q, const float* K, const float* V, const float* A, int64_t N, int T,
                     int D, int H, float scale, int round_dO, float* dQ, float* dK, float* dV, float* part,
                     float* colsums, float* cws, hipStream_t s, float* dS = nullptr);
// bf16 models: dX[n][t] (all T tokens) from the rank-one key and value
// gradients plus dY0 on the last token; false when no kernel is built for the shape
// WkT, WvT: fragment-packed bf16 copies of Wk^T and Wv^T (RJ_PACKT of the [D][D] masters)
bool dx_rank1_built(int T, int D, int H);
bool launch_dx_rank1(const float* q, const float* dO, const float* dS, const float* A, const uint4* WkT,
                     const uint4* WvT, const float* dY0, int64_t N, int T, int D, int H, float scale, float* dX,
                     hipStream_t s);
int64_t attn_bwd_part_floats(int64_t N, int T, int D, int H);
// bf16 models: dWk, dWv (written, [D][D]) from the rank-one key and value
// gradients of the last query row and the token rows X (bf16, [N][T][D]);
// ws: kv_wgrad_ws_floats(N, T, D, H) floats; false (nothing launched) when the shape
// is not built, the workspace is short or a pointer is not 16-byte aligned
bool kv_wgrad_built(int T, int D, int H);
int64_t kv_wgrad_ws_floats(int64_t N, int T, int D, int H);
// X: the token rows' byte-embedding part (bf16, [N][T][D]), or NULL with win (the
// window bytes, [N][T g]) and E (the bf16 embedding copy, [256][e]): the rows are
// gathered in the kernel.  kv_wgrad_ready: whether launch_kv_wgrad takes the shape
// with its rows gathered (pointers from the device allocator; dWv must follow
// dWk, dWv = dWk + D D)
bool kv_wgrad_ready(int64_t N, int T, int D, int H, int e, int64_t ws_cap);
bool launch_kv_wgrad(const uint16_t* X, const uint8_t* win, const uint16_t* E, int e, int g, const float* dS,
                     const float* A, const float* q, const float* dO, int64_t N, int T, int D, int H, float scale,
                     float* ws, int64_t ws_cap, float* dWk, float* dWv, hipStream_t s);
// sums over windows of the rank-one key and value gradients of the last query
// row, of dQ and of dY0 into colsums [2 T + 2][D] (sK [T][D], sV [T][D], sQ, sY);
// part: rank1_sums_part_floats floats (at most attn_bwd_part_floats); false when
// the shape is not taken
int64_t rank1_sums_part_floats(int64_t N, int T, int D);
bool launch_rank1_sums(const float* dS, const float* q, const float* A, const float* dO, const float* dQ,
                       const float* dY0, int64_t N, int T, int D, int H, float scale, int round_dO, float* part,
                       float* colsums, float* cws, hipStream_t s);
void launch_pos_table_grad(const float* sKV, const float* sQ, const float* sY, const float* Wq, const float* Wk,
                           const float* Wv, int T, int D, int rb, float* dP, hipStream_t s);
void launch_add(float* y, const float* x, int64_t rows, int64_t cols, int64_t ldy, int64_t ldx, hipStream_t s);
// dE[v][:] = sum of the e-vectors of dX (viewed as [N*W][e]) at the positions
// whose window byte is v; N*W < 2^31; deterministic
int64_t embed_bwd_ws_floats(int64_t M, int e);  // M = N * W positions
void launch_embed_bwd(const uint8_t* win, const float* dX, int64_t N, int W, int e, float* dE, float* ws,
                      hipStream_t s);
void launch_gather_kept(bool bf, const uint8_t* win, int64_t N, const void* E, int T, int D, int e, int g, void* X,
                        hipStream_t s);
// bf16, the last token of each window only: X [N][D]; false (nothing launched)
// unless e is a multiple of 8 and E, X are 16-byte aligned
bool launch_gather_last(const uint8_t* win, int64_t N, const uint16_t* E, int T, int D, int e, int g, uint16_t* X,
                        hipStream_t s);
// dW[i][j] += sum_{u < nt} P[t0 + u][i] * S[u][j]  (P: operand copy [T][D])
void launch_pos_grad(bool bf, const void* P, const float* S, int t0, int nt, int D, float* dW, hipStream_t s);
// up to three positional parts (launch_pos_grad's (S, t0, nt, dW)) in one launch
void launch_pos_grad3(bool bf, const void* P, const float* const* S, const int* t0, const int* nt, float* const* dW,
                      int njobs, int D, hipStream_t s);
void launch_adam(float* theta, const float* grad, float* m, float* v, int64_t n, float lr, float b1, float b2,
                 float eps, float bc1, float bc2, hipStream_t s, hipEvent_t t0 = nullptr, hipEvent_t t1 = nullptr);

// ---- stacked layers (layers.hip) ----
void launch_tokens(bool bf, const WinArgs& w, const void* E, const void* P, int T, int D, int e, int g, float* X,
                   hipStream_t s);
void launch_attn_rows(const float* Q, const float* K, const float* V, int64_t N, int T, int D, int H, float scale,
                      int rb, float* O, float* Akeep, hipStream_t s);
void launch_attn_bwd_rows(const float* dO, const float* Q, const float* K, const float* V, const float* A, int64_t N,
                          int T, int D, int H, float scale, int rb, float* dQ, float* dK, float* dV, hipStream_t s);
