/*
 * trace.h -- C ABI of libtrace: the batched next-byte estimator of TRACE
 * (Mao et al., "A Fast Transformer-based General-Purpose Lossless Compressor",
 * arXiv 2203.16114) and its controller-gated online update, on one AMD
 * Instinct MI355X (gfx950).
 *
 * The paper states the problem as three model calls inside its dynamic
 * compression loop (Sec. 3.2, Algorithm 1): Model.initialize(), the forward
 * estimate P(x_i | x_{i-c} .. x_{i-1}) and Model.backward on the byte just
 * coded; and one controller call that turns the step's cross-entropy into a
 * back-propagate / skip decision (Sec. 4.4, Algorithm 2, Eq. 7).  The entry
 * points below are those calls for B independent byte streams at once.
 *
 * Conventions for every call:
 *   - the return value is 0 (TRACE_OK) or a negative TRACE_E* code; nothing
 *     throws across the ABI; trace_last_error() describes the last failure of
 *     the calling thread;
 *   - "device pointer" means memory on the HIP device the model was created
 *     on; "host pointer" means ordinary CPU memory;
 *   - buffers passed in are owned by the caller and are never freed or kept
 *     by the library past the call, except where stated;
 *   - GPU work is enqueued on the caller's stream (a hipStream_t passed as
 *     void*; NULL is the legacy default stream) and is asynchronous unless the
 *     call says it synchronises; argument errors are reported synchronously,
 *     before anything is enqueued; launch failures come back as TRACE_EHIP;
 *   - one model is used by one host thread at a time.
 */
#ifndef TRACE_H
#define TRACE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
  TRACE_OK = 0,
  TRACE_EINVAL = -1,       /* bad argument or configuration                     */
  TRACE_ENOMEM = -2,       /* device or host allocation failed                  */
  TRACE_EHIP = -3,         /* a HIP runtime call or kernel launch failed        */
  TRACE_ESTATE = -4,       /* call out of order (e.g. adapt with no kept batch) */
  TRACE_ENONFINITE = -5,   /* a NaN/Inf cross-entropy reached the controller    */
  TRACE_EUNSUPPORTED = -6  /* shape valid but no kernel is built for it         */
};

enum { TRACE_FP32 = 0, TRACE_BF16 = 1 };  /* BF16: fp32 master + bf16 operand copies */
/* Flags of trace_forward_bits.
 *   TRACE_KEEP_ACTS   keep the batch's activations for trace_adapt_step
 *   TRACE_TOKEN_ATTN  run every window through the per-token attention kernel,
 *                     whose result for a window is the same bit for bit in
 *                     every launch (any n_streams, n_steps, pos0, chunking):
 *                     the step cross-entropies of a launch over many steps then
 *                     equal those of one-step launches, which a loop that may
 *                     update between steps needs for exact decisions */
enum { TRACE_KEEP_ACTS = 1u, TRACE_TOKEN_ATTN = 2u };

/* Model shape and optimiser settings.
 *   W        window bytes, the c*g bytes before the target (Sec. 4.2; Alg. 1 line 8)
 *   e        per-byte embedding width h/g (Sec. 4.2)
 *   g        bytes per group; T = W/g tokens of width d = g*e (Sec. 4.2, Fig. 4b)
 *   H        attention heads, head width d/H (Eqs. 1-2)
 *   F        FFN width (Eq. 3)
 *   k        shared-FFN repeats N (Sec. 4.3, Fig. 4c)
 *   dtype    TRACE_FP32: every GEMM operand in fp32; TRACE_BF16: GEMM operands
 *            (weights and activations) rounded to bf16 (RNE), fp32 accumulate,
 *            fp32 residual stream, softmax, code lengths, master weights, Adam
 *   use_pos  1: a learned positional table P[T][d] is added after grouping
 *   max_windows  windows per internal forward chunk (workspace size); a
 *            forward over more windows runs in chunks, with identical results
 *   max_keep windows a KEEP_ACTS forward may hold for trace_adapt_step
 *            (0: the model cannot adapt)
 *   lr, beta1, beta2, eps  Adam (Sec. 6 uses lr 0.001)
 * Supported shapes: W % g == 0, d % H == 0, T in {4, 8}, d/H in {32, 64},
 * d in {64, 128, 256, 512} (a multiple of 64), e % 8 == 0, e <= 128, F % 256 == 0,
 * 1 <= k <= 8.  Others return TRACE_EINVAL or TRACE_EUNSUPPORTED. */
typedef struct {
  int32_t W, e, g, H, F, k;
  int32_t dtype;
  int32_t use_pos;
  int64_t max_windows;
  int64_t max_keep;
  double lr, beta1, beta2, eps; /* used as float, except beta^t in double for the bias corrections */
  /* 0: the k repeats of Eq. 3 share W1, W2 (Sec. 4.3); 1: each repeat has its
   * own (the deep-FFN variant of Sec. 6.3): W1 and W2 in the flat order become
   * k consecutive blocks, repeat r's at r * D * F. */
  int32_t untied_ffn;
  /* TRACE_ATTN_SOFTMAX: Eqs. 1-2; TRACE_ATTN_PERFORMER: the FAVOR+ attention of
   * the Performer the paper's experiments use as backbone (Sec. 6), forward
   * only, with n_features positive random features (0: 128 for d/H = 32, 256
   * for 64; a multiple of 16, at most 512) whose projection is set by
   * trace_set_features before the first forward. */
  int32_t attention;
  int32_t n_features;
  /* layers of Eq. 4 stacked (Sec. 6.3, Fig. 7; 0 or 1: one layer, the
   * estimator of the workloads), at most 8; each has its own Wq, Wk, Wv, Wo,
   * W1, W2, stored in the flat order as `layers` consecutive blocks of each
   * (layer l's Wq at l * d * d within Wq's span).  Layer 0 reads the tokens
   * X = E + P; later layers read the previous layer's output, rounded like an
   * FFN input in bf16 models.  Softmax attention only. */
  int32_t layers;
  int32_t reserved_; /* 0 */
} trace_config;

enum { TRACE_ATTN_SOFTMAX = 0, TRACE_ATTN_PERFORMER = 1 };

typedef struct trace_model trace_model; /* opaque, library-owned */

/* Allocates a model on the current HIP device: fp32 master parameters in the
 * canonical flat order E[256][e], P[T][d], Wq, Wk, Wv, Wo [d][d], W1 [d][F],
 * W2 [F][d], Wout [d][256], bout [256] (every matrix row-major [in][out]),
 * Adam moments, operand copies and workspace.  Parameters start at zero until
 * trace_init_weights.  EINVAL for an invalid config, EUNSUPPORTED for a shape
 * with no kernel, ENOMEM if device memory runs out.  *out is NULL on error. */
int trace_create(const trace_config* cfg, trace_model** out);
void trace_destroy(trace_model* m); /* NULL is a no-op; synchronises the device */

/* Number of parameters (flat master length) of a configuration; host only. */
int trace_param_count(const trace_config* cfg, int64_t* n);

/* Model.initialize() of Alg. 1: the dynamic setting starts from a random
 * model (Sec. 3.2, Sec. 5 "Dynamic-Random").  With host_flat == NULL every
 * entry of E, P, Wq .. Wout is std * N(0, 1), drawn in flat order by
 * Box-Muller (cos, then sin) from splitmix64 uniforms ((x >> 11) + 0.5) * 2^-53
 * seeded with `seed`, computed in double and rounded to float; bout = 0.
 * With host_flat != NULL (a host array of trace_param_count floats) it is
 * copied instead.  Resets Adam (m = v = 0, step count 0) and drops any kept
 * batch.  Synchronises the device. */
int trace_init_weights(trace_model* m, uint64_t seed, double std, const float* host_flat);

/* The random projection of the Performer's positive random features (Sec. 6's
 * backbone; FAVOR+): omega[i][c] (host, row-major [n_features][d/H] floats),
 * one for all heads.  With q' = q (d/H)^-1/4 and k' = k (d/H)^-1/4 per head,
 * the last query row's weight on key u is phi(q')^T phi(k'_u) normalised over
 * u, phi(x) = exp(omega x - |x|^2/2) (the 1/sqrt(m) factor cancels); the
 * projections are formed in fp32 (bf16 models: omega rounded to bf16, the
 * projected vector split into two bf16 parts).  Copies omega (synchronises);
 * EINVAL unless the model uses TRACE_ATTN_PERFORMER and n = n_features * d/H. */
int trace_set_features(trace_model* m, const float* host_omega, int64_t n);

/* The same generator into a host array of n = trace_param_count floats,
 * without a model or a GPU. */
int trace_init_flat_host(const trace_config* cfg, uint64_t seed, double std, float* host_out, int64_t n);

/* Model.forward of Alg. 1 line 8 for many streams and steps at once, with the
 * code length of Alg. 2 line 3.  Window (b, s), b < n_streams, s < n_steps,
 * is d_streams[b*stride + pos0 + s - W .. b*stride + pos0 + s - 1] (oldest
 * first) and its target is the byte d_streams[b*stride + pos0 + s]; requires
 * pos0 >= W.  Writes
 *   d_bits[b*n_steps + s]            = -log2 p(target)            (device, fp32)
 *   d_logits[(b*n_steps + s)*256+v]  = head output z_v            (device, fp32; optional)
 *   d_step_ce[s] = mean over b of d_bits[b*n_steps + s]           (device, fp64; optional)
 * The byte-grouped single-layer transformer is: tokens by byte grouping
 * (Sec. 4.2), causal multi-head attention (Eqs. 1-2), the layer of Eq. 4 with
 * its FFN (Eq. 3) shared and applied k times (Sec. 4.3), and a 256-way softmax
 * head reading the last token.  flags may hold TRACE_KEEP_ACTS: the call then
 * also keeps the activations of these n_streams*n_steps <= max_keep windows
 * for trace_adapt_step; TRACE_TOKEN_ATTN as above.  For a given attention
 * kernel, results depend only on each window's bytes and the weights (not on
 * n_streams, n_steps, chunking or position in the batch).  bf16 launches whose
 * 64-window tiles each lie in one stream (n_steps and the first window a
 * multiple of 64), without TRACE_TOKEN_ATTN, share byte groups between windows
 * in a kernel whose sums are ordered differently: their results agree with the
 * other launches' within rounding, not bit for bit. */
int trace_forward_bits(trace_model* m, const uint8_t* d_streams, int64_t stride, int32_t n_streams,
                       int64_t pos0, int32_t n_steps, float* d_bits, float* d_logits,
                       double* d_step_ce, uint32_t flags, void* stream);

/* Model.backward of Alg. 1 line 10 on the batch kept by the last
 * KEEP_ACTS forward (softmax attention only: EUNSUPPORTED for a Performer
 * model): the gradient of the batch-mean cross-entropy (nats)
 * followed by one Adam step (Kingma & Ba, Alg. 1; bias-corrected; the step
 * count advances once per call) on the fp32 master, then a refresh of the
 * operand copies.  The kept batch is consumed.  ESTATE if none is kept. */
int trace_adapt_step(trace_model* m, void* stream);

/* The back-prop controller of Sec. 4.4 (Algorithm 2, uniform weights, Eq. 7):
 * a FIFO loss cache of the last t step cross-entropies (bits) and their sum.
 * decide(e) sets *update = 1 (back-propagate) iff fewer than t values are
 * cached yet, or e > sum/t + delta in IEEE double; then the oldest value
 * leaves a full cache and e enters it, whatever the decision.  Host only,
 * O(1), no GPU.  A non-finite e returns ENONFINITE with *update = 0 and leaves
 * the cache unchanged. */
/* The forward of trace_forward_bits (same arguments, flags and results, bit
 * for bit) for callers that cannot allocate device memory: code under HIP graph
 * capture, serving loops, harnesses that forbid allocation.  Its only device
 * workspace, the hand-off between the attention and FFN kernels
 * (n_streams * n_steps * d floats), lives in one fixed 32 MiB array that the
 * library holds on each device from its first trace_create there until the
 * process ends; the call allocates nothing and records no timing events.
 * The batch must fit that array in one launch: n_streams * n_steps * d * 4 <=
 * 32 MiB (e.g. 32768 windows at d = 256), else EINVAL before any work.  Every
 * call on a device shares the array, so calls that overlap on one device (two
 * streams, two threads) race; calls queued on one stream do not.  The model's
 * device must be current. */
int trace_forward_bits_noalloc(trace_model* m, const uint8_t* d_streams, int64_t stride, int32_t n_streams,
                               int64_t pos0, int32_t n_steps, float* d_bits, float* d_logits, double* d_step_ce,
                               uint32_t flags, void* stream);

typedef struct {
  int32_t t, count, head, pad_;
  double delta, sum;
  double ring[256];
} trace_controller;
int trace_controller_init(trace_controller* c, int32_t t, double delta); /* 1 <= t <= 256 */
int trace_controller_decide(trace_controller* c, double batch_ce_bits, int32_t* update);

/* Alg. 1 with the controller of Alg. 2 on the model's estimated code lengths,
 * for n_streams streams over steps s < n_steps (target position pos0 + s, as
 * in trace_forward_bits): each step forms the estimates of the n_streams
 * windows and the step cross-entropy e_s (mean bits, fp64); then, by mode,
 * 0: no update, 1: the controller of Alg. 2 (t = ctl_t, delta = ctl_delta, as
 * trace_controller_decide) decides, 2: always; an update runs the backward and
 * Adam step of trace_adapt_step on that step's batch before step s + 1.
 * Forwards run ahead over up to max_spec steps at unchanged weights; the
 * controller walks their cross-entropies and the first step it flags is run
 * again keeping activations and updated, the walk resuming after it.  Every
 * forward uses TRACE_TOKEN_ATTN, so the cross-entropies, decisions and final
 * state are bit for bit those of a loop of one-step forwards (max_spec = 1).
 * Outputs (host, each may be NULL): step_ce[n_steps] (bits), decisions[n_steps]
 * (0/1), *n_updates.  Requires n_streams <= max_keep when mode != 0.  The
 * model's weights and Adam state advance with the updates.  Allocates its
 * buffers for the call (device: n_streams*max_spec floats and n_steps doubles;
 * pinned host: n_steps doubles) and synchronises the stream before returning. */
int trace_gated_run(trace_model* m, const uint8_t* d_streams, int64_t stride, int32_t n_streams, int64_t pos0,
                    int32_t n_steps, int32_t mode, int32_t ctl_t, double ctl_delta, int32_t max_spec,
                    double* step_ce, int32_t* decisions, int64_t* n_updates, void* stream);

/* Copies of the training state (host arrays of trace_param_count floats each;
 * any pointer may be NULL to skip it).  get synchronises the device; set also
 * refreshes the operand copies and drops any kept batch. */
int trace_get_state(trace_model* m, float* theta, float* adam_m, float* adam_v, int64_t* step, int64_t n);
int trace_set_state(trace_model* m, const float* theta, const float* adam_m, const float* adam_v, int64_t step,
                    int64_t n);

/* Gradient (flat, canonical order) computed by the last trace_adapt_step,
 * copied to a host array of trace_param_count floats; synchronises. */
int trace_get_grads(trace_model* m, float* host_out, int64_t n);

/* ---------------------------------------------------------------- coding ----
 * Alg. 1, lines 3 and 9: the first W bytes of a stream are coded with
 * probability 1/256, every later byte with the model's estimate.  The paper
 * names arithmetic coding and does not fix how the estimate becomes integer
 * intervals; this library uses:
 *   frequencies (trace_quantize): for logits z[256] of a window, m = max z,
 *     d_s = (m - z_s) * log2(e) in float32 (two IEEE operations), u_s =
 *     trunc(256 d_s + 0.5) (float32) or 32*256-1 if d_s >= 32 (or NaN),
 *     w_s = T[u_s % 256] >> (u_s / 256), freq_s = 1 + (65280 w_s) / sum w
 *     (integer division); T as trace_quant_table.  Every freq_s >= 1 and the
 *     total is at most 65536;
 *   the coder: a 32-bit range coder (integer renormalisation by bytes, carry
 *     into the byte held back); a code starts with byte 0, and its decoder
 *     reads zeros past the end.
 * Both directions of the compressor run the same launches in the same order,
 * so the decoder sees bit for bit the encoder's frequencies. */

/* T[j] = round(2^31 * 2^(-j/256)), j < 256, into out[256] (host). */
int trace_quant_table(uint32_t* out);

/* Frequencies of n windows: d_freq[w*256 + s] (device uint16, 8-byte
 * aligned) from d_logits[w*256 + s] (device fp32, 16-byte aligned), on the
 * stream; n = 0 is a no-op. */
int trace_quantize(const float* d_logits, int64_t n, uint16_t* d_freq, void* stream);

/* One code (host) for sym[i] under frequency row freq[i*freq_stride ..
 * +256] (each >= 1, total <= 65536), or under 1/256 when freq_stride = 0.
 * Writes at most cap bytes to out and the code length to *size; EINVAL if cap
 * is too small (then *size is the length needed). */
int trace_rc_encode(const uint16_t* freq, int64_t freq_stride, const uint8_t* sym, int64_t n, uint8_t* out,
                    int64_t cap, int64_t* size);
/* Inverse of trace_rc_encode: n symbols of the code in[0 .. size) (host). */
int trace_rc_decode(const uint16_t* freq, int64_t freq_stride, const uint8_t* in, int64_t size, int64_t n,
                    uint8_t* sym_out);

/* The compressor of Alg. 1 over n_streams streams of `length` bytes each,
 * stream b at d_streams[b*stride ..] (device).  One code per stream: stream
 * b's goes to out[b*out_stride ..] (host) and its length to out_sizes[b].
 * At each position i >= W: one forward over the n_streams windows ending
 * before i (trace_forward_bits, one step), frequencies (trace_quantize), the
 * byte at i coded; then, by mode, 0: no update, 1: the controller of Alg. 2
 * (trace_controller_*, t = ctl_t, delta = ctl_delta) on the batch mean of the
 * coded lengths log2(total) - log2(freq[x]) (double, streams in order),
 * 2: always; an update re-runs that forward keeping activations and calls
 * trace_adapt_step (Alg. 1, line 10).  The model's weights and Adam state
 * advance as in the loop; *n_updates (may be NULL) counts updates.
 * n_streams <= max_windows, and <= max_keep when mode != 0.  EINVAL if a code
 * does not fit out_stride (out_sizes then hold the lengths needed); a code
 * takes at most about 2 bytes per byte. */
int trace_compress(trace_model* m, const uint8_t* d_streams, int64_t stride, int32_t n_streams, int64_t length,
                   int32_t mode, int32_t ctl_t, double ctl_delta, uint8_t* out, int64_t out_stride,
                   int64_t* out_sizes, int64_t* n_updates, void* stream);
/* Inverse of trace_compress, for a model in the state the encoder's started
 * from: codes at comp[b*comp_stride ..] of comp_sizes[b] bytes (host); the
 * bytes go to d_out[b*stride ..] (device, stride >= length), byte by byte as
 * they are decoded, with the same forwards, controller and updates. */
int trace_decompress(trace_model* m, const uint8_t* comp, int64_t comp_stride, const int64_t* comp_sizes,
                     int32_t n_streams, int64_t length, int32_t mode, int32_t ctl_t, double ctl_delta,
                     uint8_t* d_out, int64_t stride, int64_t* n_updates, void* stream);

/* One product of the update step on the bf16 GEMM kernels alone (test
 * support): C[m][n] = sum_k A(m,k) B(k,n), all device memory, C row-major
 * [M][N].  A(m,k) is d_A[m*K + k] when a_kc, else d_A[k*M + m]; B(k,n) is
 * d_B[n*K + k] when b_kc, else d_B[k*N + n].  mode_a / mode_b: 0 fp32 rounded
 * to bf16 as it is read, 1 fp32 split into bf16 hi + lo (two products; not both
 * operands), 2 bf16 elements.  half_c: C written as bf16 (no split over k).
 * kernel: 1 the 128-tile kernel, 2 the 256-tile kernel.  d_ws holds ws_floats
 * floats of split-K partial sums (fewer splits when it is small).  EUNSUPPORTED
 * when the operands do not fit the kernel's vector reads (fp32: a multiple of 4
 * along the contiguous dimension; bf16: K a multiple of 8 when k is contiguous,
 * a multiple of 4 rows otherwise; 16-byte aligned pointers). */
int trace_debug_gemm(int M, int N, int K, const void* d_A, int a_kc, int mode_a, const void* d_B, int b_kc,
                     int mode_b, void* d_C, int half_c, int kernel, float* d_ws, int64_t ws_floats, void* stream);

/* Byte-group gather of the update step (Sec. 4.2; test support): for the batch
 * kept by the last KEEP_ACTS forward (window bytes as the attention kernel kept
 * them), writes the byte-embedding part of every token with the kernel
 * trace_adapt_step uses, d_X[(n*T + t)*d + j*e + c] = E[byte j of group t of
 * window n][c] (device; fp32 for TRACE_FP32 models, the bf16 bit patterns of
 * the operand copy for TRACE_BF16 models; n = b*n_steps + s of that forward).
 * The positional table is not added (the update adds its part separately).
 * ESTATE if no batch is kept; the kept batch stays kept. */
int trace_debug_kept_tokens(trace_model* m, void* d_X, void* stream);

/* Test support for the key and value weight gradients of bf16 models (the
 * rank-one rows of the last query row, Eq. 2's attention; Alg. 1 line 10):
 * recomputes dWk and dWv from the buffers the last trace_adapt_step left (its
 * score gradients, attention weights, q and dO; the window bytes of its batch;
 * the current embedding copy) twice, into d_rows from the token rows written
 * by the update's gather (trace_debug_kept_tokens' kernel), into d_gathered
 * with the rows gathered inside the weight-gradient kernel.  Each output is
 * [2][d][d] fp32 (dWk, then dWv), device memory owned by the caller; the model's
 * gradient is not touched.  The two are meant to be bitwise equal.  ESTATE
 * before the first update; EUNSUPPORTED for fp32 models and shapes the kernel
 * does not take (the path that uses it then is the GEMM over every token row). */
int trace_debug_kv_wgrad(trace_model* m, float* d_gathered, float* d_rows, void* stream);

/* Per-kernel timing with HIP events recorded on the caller's stream around each
 * launch (measurement support; off by default).  While enabled, every kernel
 * launch of the calls above is bracketed by two events (the Adam kernel's
 * dispatch records its two itself, so that region is the kernel's own start to
 * end, without the gap an event pair around one short launch adds; the other
 * kinds span all their kernels' launches); trace_read_timing waits
 * for them, returns per-kind totals (milliseconds) and launch counts in arrays
 * of TRACE_NKINDS entries, and starts a new measurement.  Every 65536 regions
 * the recorded ones are folded into the totals, which waits for the GPU (only
 * while timing is on); overflow counts regions lost to a failed event read. */
enum {
  TRACE_KIND_ATTN = 0,      /* fused gather + attention block                 */
  TRACE_KIND_FFN_HEAD = 1,  /* fused shared FFN x k + softmax head            */
  TRACE_KIND_STEP_CE = 2,   /* per-step mean code length                      */
  TRACE_KIND_BACKWARD = 3,  /* gradient of one gated update (all its kernels) */
  TRACE_KIND_ADAM = 4,      /* the Adam update                                */
  TRACE_KIND_REFRESH = 5,   /* operand copies refreshed from the master       */
  TRACE_NKINDS = 6
};
int trace_set_timing(trace_model* m, int enable);
int trace_read_timing(trace_model* m, double* ms_total, int64_t* launches, int64_t* overflow);

const char* trace_strerror(int code);
const char* trace_last_error(void); /* thread-local text of the last failure ("" if none) */

#ifdef __cplusplus
}
#endif
#endif /* TRACE_H */
