// C ABI of libtrace (include/trace.h): device memory, operand copies and the
// launch sequence of the forward estimator and of the gated update.
#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <cmath>
#include <array>
#include <cstring>
#include <string>
#include <vector>

#include "../../include/trace.h"
#include "host.h"
#include "kernels.h"

struct trace_model {
  trace_config cfg;
  Layout L;
  bool bf;
  int device;
  attn_fn attn;
  ffn_fn ffn;
  int64_t max_windows, max_keep;
  // fp32 master, Adam moments, gradient (canonical flat order)
  float *theta, *am, *av, *grad;
  int64_t step;
  bool upd_run;  // trace_adapt_step has run in this process (its backward buffers hold values)
  // operand copies
  void *Ec, *Pc;
  float* PW;  // [3][T][D] positional parts of the q, k, v projections
  uint4 *Wq, *Wk, *Wv, *Wo, *W1, *W2, *Wout;
  uint4 *WkT, *WvT;  // bf16 models that keep activations: packed Wk^T, Wv^T (input gradient of the tokens)
  // bf16 models that keep activations: the master's Wq .. Wout range as bf16
  // operand values, same order (B operands of the update's products)
  uint16_t* Wh;
  // Performer attention: packed random projection (device), features, set yet
  uint4* Om;
  int nfeat;
  bool feats_set;
  // forward workspace
  float* h0;
  // stacked layers: the lower layers' forward buffers (per chunk of lcap
  // windows) and split-K workspace; kept activations of every lower layer
  // (klX: the input of every layer, the top's included) and their backward
  // buffers
  int64_t lcap, fws_cap;
  float *lx[2], *lq, *lk, *lv, *lo, *ly[2], *lu, *lg, *fws;
  float *klX, *klQ, *klK, *klV, *klA, *klO, *klY, *klU;
  float *ldY, *ldU, *ldG, *ldO, *ldQ;
  // kept batch
  bool kept;
  int64_t keepN;
  uint8_t* kwin;
  int32_t* ktgt;
  float *kq, *kK, *kV, *kA, *kO, *kY, *kU, *kZ;
  uint16_t* kG;  // bf16 models: GELU(U) of each repeat as bf16 operand values
  // backward scratch
  // dY: gradients w.r.t. the k+1 residual states, dU: w.r.t. the k pre-GELU
  // activations (one buffer per repeat, read by the weight gradients later);
  // in bf16 models dU, Xk (the byte-embedding part of the kept tokens) and the
  // kept Y hold bf16 elements: all are only read as bf16 operands
  float *dz, *dY, *dU, *G, *dO, *dQ, *dK, *dV, *dX, *Xk, *sP, *gws, *cws, *ews, *apart;
  float* dSc;  // [N][H][T] gradients of the last row's attention scores
  int64_t gws_cap;
  // second stream of the update step (the weight-gradient branch), its own
  // split-K and column-sum workspaces, and the events that order the two streams
  hipStream_t side;
  float *gws2, *cws2;
  std::vector<hipEvent_t> sev;
  size_t sev_next;
  std::vector<void*> allocs;
  // event timing (trace_set_timing)
  bool timing;
  std::vector<hipEvent_t> events;
  size_t ev_used;
  std::vector<int> ev_kind;  // kind of the launch bracketed by events 2i, 2i+1
  int64_t overflow;
  double t_ms[TRACE_NKINDS];  // regions already folded in (see harvest)
  int64_t t_n[TRACE_NKINDS];
};

namespace {

int fail(int code, const std::string& msg) {
  trace_set_error(msg);
  return code;
}

int hip_fail(hipError_t e, const char* where) {
  return fail(TRACE_EHIP, std::string(where) + ": " + hipGetErrorString(e));
}

template <typename P>
bool dalloc(trace_model* m, P** p, int64_t bytes) {
  void* q = nullptr;
  if (bytes <= 0) bytes = 16;
  if (hipMalloc(&q, (size_t)bytes) != hipSuccess) {
    *p = nullptr;
    return false;
  }
  m->allocs.push_back(q);
  *p = (P*)q;
  return true;
}

void free_all(trace_model* m) {
  for (void* p : m->allocs) (void)hipFree(p);
  m->allocs.clear();
  for (hipEvent_t e : m->events) (void)hipEventDestroy(e);
  m->events.clear();
  for (hipEvent_t e : m->sev) (void)hipEventDestroy(e);
  m->sev.clear();
  if (m->side) (void)hipStreamDestroy(m->side);
  m->side = nullptr;
}

// An event marking everything issued so far on stream `from`.  A wait applies
// to the record made before it, so the events are reused round-robin; every
// mark is waited for within a few marks of being made.
hipEvent_t mark(trace_model* m, hipStream_t from) {
  hipEvent_t e = m->sev[m->sev_next];
  m->sev_next = (m->sev_next + 1) % m->sev.size();
  (void)hipEventRecord(e, from);
  return e;
}
void after(hipStream_t to, hipEvent_t e) { (void)hipStreamWaitEvent(to, e, 0); }
// Work on stream `to` after everything issued so far on stream `from`.
void order(trace_model* m, hipStream_t from, hipStream_t to) { after(to, mark(m, from)); }

// The GEMM shapes (M, N, K) of trace_adapt_step for N kept windows.
std::vector<std::array<int, 3>> adapt_gemm_shapes(const trace_model* m, int64_t N) {
  const int D = m->L.D, F = m->cfg.F, T = m->L.T;
  const int n = (int)N;
  std::vector<std::array<int, 3>> v = {{D, 256, n}, {n, D, 256}, {F, D, n},     {n, F, D},
                                       {D, F, n},   {n, D, F},   {D, D, n},     {n, D, D},
                                       {D, D, n * T}, {n * T, D, D}, {n * T, D, 2 * D}};
  if (m->cfg.k > 1) {  // the FFN weight gradients summed over the repeats in one product
    v.push_back({F, D, m->cfg.k * n});
    v.push_back({D, F, m->cfg.k * n});
  }
  if (m->L.NL > 1) {  // the lower layers' products run over every token row
    const int r = n * T;
    for (std::array<int, 3> x : std::vector<std::array<int, 3>>{
             {r, F, D}, {F, D, r}, {D, F, r}, {r, D, F}, {D, D, r}, {r, D, D}})
      v.push_back(x);
  }
  return v;
}
// Largest split-K workspace (floats) over those GEMMs, for either GEMM path.
int64_t adapt_gemm_ws(const trace_model* m, int64_t N) {
  int64_t w = 0;
  for (auto& s : adapt_gemm_shapes(m, N))
    w = std::max(w, std::max(gemm_ws_floats(s[0], s[1], s[2]), bgemm_ws_floats(s[0], s[1], s[2])));
  if (m->bf) w = std::max(w, kv_wgrad_ws_floats(N, m->L.T, m->L.D, m->cfg.H));
  return w;
}

hipStream_t S(void* s) { return (hipStream_t)s; }

constexpr size_t MAX_TIMED = 65536;

// Folds every recorded region into the per-kind totals (waiting for each
// region's end) and frees the events for reuse; false if a HIP call failed.
bool harvest(trace_model* m) {
  bool ok = true;
  for (size_t i = 0; i < m->ev_kind.size(); ++i) {
    const int kind = m->ev_kind[i];
    if (kind < 0) continue;
    hipError_t e = hipEventSynchronize(m->events[2 * i + 1]);
    float ms = 0.f;
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, m->events[2 * i], m->events[2 * i + 1]);
    if (e != hipSuccess) {
      ok = false;
      continue;
    }
    m->t_ms[kind] += ms;
    m->t_n[kind] += 1;
  }
  m->ev_kind.clear();
  m->ev_used = 0;
  return ok;
}

// Reserves a timed region (two events); returns its index or -1.  When all
// MAX_TIMED regions are in use, the recorded ones are folded into the totals
// first (a wait for the GPU; only while timing is on).
long treserve(trace_model* m) {
  if (!m->timing) return -1;
  if (m->ev_kind.size() >= MAX_TIMED && !harvest(m)) {
    m->overflow += 1;
    return -1;
  }
  while (m->events.size() < m->ev_used + 2) {
    hipEvent_t e;
    if (hipEventCreate(&e) != hipSuccess) return -1;
    m->events.push_back(e);
  }
  const long i = (long)m->ev_kind.size();
  m->ev_used += 2;
  m->ev_kind.push_back(-1);
  return i;
}
// Starts a timed region of `kind` on stream s; returns its index or -1.
long tbegin(trace_model* m, hipStream_t s) {
  const long i = treserve(m);
  if (i >= 0) (void)hipEventRecord(m->events[2 * i], s);
  return i;
}
void tend(trace_model* m, long i, int kind, hipStream_t s) {
  if (i < 0) return;
  (void)hipEventRecord(m->events[2 * i + 1], s);
  m->ev_kind[i] = kind;
}

// Refresh the operand copies from the fp32 master (one launch).
bool refresh_operands(trace_model* m, hipStream_t s) {
  const long tk = tbegin(m, s);
  const Layout& L = m->L;
  const int D = L.D, F = m->cfg.F;
  const float* th = m->theta;
  const bool pos = m->cfg.use_pos != 0;
  auto job = [](int kind, const float* src, void* dst, int64_t K, int N, float scale = 1.f) {
    RefreshJob j;
    j.src = src;
    j.src2 = nullptr;
    j.dst = dst;
    j.kind = kind;
    j.K = (int)K;
    j.N = N;
    j.use_pos = 0;
    j.scale = scale;
    return j;
  };
  // the fused kernels run the top layer (the only layer when NL = 1); with
  // stacked layers its input carries no positional part, so P.W is zero
  const int top = L.NL - 1;
  RefreshJob pt = L.NL > 1 ? job(RJ_ZERO, nullptr, m->PW, 3 * (int64_t)L.T * D, 0)
                           : job(RJ_PTAB, th + L.off[P_P], m->PW, L.T, D);
  if (L.NL == 1) {
    pt.src2 = th + L.off[P_WQ];  // W_q, W_k, W_v are consecutive D x D blocks of the master
    pt.use_pos = pos;
  }
  // the positional table's blocks run longest: they are dispatched first
  const RefreshJob jobs[] = {
      pt,
      job(RJ_PACK, th + L.at(P_W1, top), m->W1, D, F),
      // bf16: W2/2 (exact), since the bf16 FFN kernel forms 2 GELU(U) (exact in bf16 too)
      job(RJ_PACK, th + L.at(P_W2, top), m->W2, F, D, m->bf ? 0.5f : 1.f),
      job(RJ_PACK, th + L.at(P_WQ, top), m->Wq, D, D),
      job(RJ_PACK, th + L.at(P_WK, top), m->Wk, D, D),
      job(RJ_PACK, th + L.at(P_WV, top), m->Wv, D, D),
      job(RJ_PACK, th + L.at(P_WO, top), m->Wo, D, D),
      job(RJ_PACK, th + L.off[P_WOUT], m->Wout, D, 256),
      job(RJ_CVT, th + L.off[P_E], m->Ec, L.size[P_E], 0),
      pos ? job(RJ_CVT, th + L.off[P_P], m->Pc, L.size[P_P], 0)
          : job(RJ_ZERO, nullptr, m->Pc, (L.size[P_P] * (m->bf ? 2 : 4) + 3) / 4, 0),
      // the update's input gradient of the tokens and the B operands of its
      // products (bf16 models that keep activations)
      job(RJ_PACKT, th + L.at(P_WK, top), m->WkT, D, D),
      job(RJ_PACKT, th + L.at(P_WV, top), m->WvT, D, D),
      job(RJ_CVT8, th + L.off[P_WQ], m->Wh, L.off[P_BOUT] - L.off[P_WQ], 0),
  };
  const int njobs = (int)(sizeof(jobs) / sizeof(jobs[0])) - (m->WkT ? 0 : 3);
  bool ok = launch_refresh(m->bf, jobs, njobs, s);
  // untied FFN: the packed copies of repeats 1 .. k-1
  const int64_t es_ = m->bf ? 2 : 4;
  for (int r = 1; ok && m->cfg.untied_ffn && r < m->cfg.k; ++r) {
    const RefreshJob more[] = {
        job(RJ_PACK, th + L.at(P_W1, top) + (int64_t)r * D * F, (char*)m->W1 + (int64_t)r * D * F * es_, D, F),
        job(RJ_PACK, th + L.at(P_W2, top) + (int64_t)r * F * D, (char*)m->W2 + (int64_t)r * F * D * es_, F, D,
            m->bf ? 0.5f : 1.f)};
    ok = launch_refresh(m->bf, more, 2, s);
  }
  tend(m, tk, TRACE_KIND_REFRESH, s);
  return ok;
}

GemmArgs gemm(int M, int N, int K, const float* A, int64_t sam, int64_t sak, int rA, const float* B, int64_t sbk,
              int64_t sbn, int rB, float* C, int64_t ldc, float beta) {
  GemmArgs g;
  g.M = M;
  g.N = N;
  g.K = K;
  g.A = A;
  g.sam = sam;
  g.sak = sak;
  g.B = B;
  g.sbk = sbk;
  g.sbn = sbn;
  g.C = C;
  g.ldc = ldc;
  g.roundA = rA;
  g.roundB = rB;
  g.beta = beta;
  g.gelu_u = nullptr;
  g.halfA = g.halfB = g.halfC = 0;
  g.Cin = nullptr;
  g.r1c = nullptr;
  g.r1tsh = g.r1dsh = g.r1H = g.r1round = 0;
  g.r1scale = 1.f;
  return g;
}

// Kept activations of lower layer l of a KEEP_ACTS forward (NULL: not kept).
struct LowerKeep {
  float *Q, *K, *V, *A, *O, *Y, *U;  // Y: inputs of the k FFN repeats; U: their pre-GELU values
  int64_t ys, us;                    // floats between repeats in Y and in U
};
LowerKeep lower_keep(const trace_model* m, int l) {
  LowerKeep k;
  const int64_t R = m->max_keep * m->L.T, D = m->L.D, F = m->cfg.F, kk = m->cfg.k;
  k.ys = R * D;
  k.us = R * F;
  k.Q = m->klQ + l * R * D;
  k.K = m->klK + l * R * D;
  k.V = m->klV + l * R * D;
  k.A = m->klA + l * m->max_keep * m->cfg.H * m->L.T * m->L.T;
  k.O = m->klO + l * R * D;
  k.Y = m->klY + l * kk * R * D;
  k.U = m->klU + l * kk * R * F;
  return k;
}

// Lower layer l (every token row) of the forward over N windows: X -> Xn,
// X and Xn [N][T][D] fp32.  The products are GEMMs on the update's kernels
// (layer 0 reads the token X = E + P as it is: split into two bf16 parts in
// bf16 models; later layers read their input rounded, a bf16 storage point).
// With kp, every intermediate the backward needs is written there.
bool lower_forward(trace_model* m, int l, const float* X, float* Xn, int64_t N, const LowerKeep* kp, hipStream_t s) {
  const Layout& L = m->L;
  const int T = L.T, D = L.D, F = m->cfg.F, H = m->cfg.H, k = m->cfg.k;
  const int rb = m->bf ? 1 : 0, rX = (l == 0) ? 0 : rb;
  const int R = (int)(N * T);
  const float* th = m->theta;
  float* ws = m->fws;
  const int64_t cap = m->fws_cap;
  float* Q = kp ? kp->Q : m->lq;
  float* K = kp ? kp->K : m->lk;
  float* V = kp ? kp->V : m->lv;
  float* O = kp ? kp->O : m->lo;
  bool ok = true;
  ok = launch_gemm(gemm(R, D, D, X, D, 1, rX, th + L.at(P_WQ, l), D, 1, rb, Q, D, 0.f), ws, cap, s) && ok;
  ok = launch_gemm(gemm(R, D, D, X, D, 1, rX, th + L.at(P_WK, l), D, 1, rb, K, D, 0.f), ws, cap, s) && ok;
  ok = launch_gemm(gemm(R, D, D, X, D, 1, rX, th + L.at(P_WV, l), D, 1, rb, V, D, 0.f), ws, cap, s) && ok;
  launch_attn_rows(Q, K, V, N, T, D, H, (float)(1.0 / std::sqrt((double)L.DH)), rb, O, kp ? kp->A : nullptr, s);
  // Y_0 = O.Wo + X, then Y_r = Y_{r-1} + G(Y_{r-1} W1) W2 (each sum: copy, then
  // a product accumulated onto it)
  const float* Yin = kp ? kp->Y : m->ly[0];
  (void)hipMemcpyAsync((void*)Yin, X, (size_t)R * D * 4, hipMemcpyDeviceToDevice, s);
  ok = launch_gemm(gemm(R, D, D, O, D, 1, rb, th + L.at(P_WO, l), D, 1, rb, (float*)Yin, D, 1.f), ws, cap, s) && ok;
  for (int r = 0; r < k; ++r) {
    const int64_t wr = m->cfg.untied_ffn ? (int64_t)r * D * F : 0;
    float* U = kp ? kp->U + r * kp->us : m->lu;
    ok = launch_gemm(gemm(R, F, D, Yin, D, 1, rb, th + L.at(P_W1, l) + wr, F, 1, rb, U, F, 0.f), ws, cap, s) && ok;
    launch_gelu_fwd_round(U, m->lg, (int64_t)R * F, rb, s);
    float* Yout = r == k - 1 ? Xn : (kp ? kp->Y + (r + 1) * kp->ys : m->ly[(r + 1) & 1]);
    (void)hipMemcpyAsync(Yout, Yin, (size_t)R * D * 4, hipMemcpyDeviceToDevice, s);
    ok = launch_gemm(gemm(R, D, F, m->lg, F, 1, rb, th + L.at(P_W2, l) + wr, D, 1, rb, Yout, D, 1.f), ws, cap, s) &&
         ok;
    Yin = Yout;
  }
  return ok;
}

// Backward of lower layer l over every token row: on entry m->dX holds the
// gradient w.r.t. the layer's output [N][T][D], on return w.r.t. its input.
// The chain of layer_backward in the oracle, with the layer's weight
// gradients written at layer l's blocks; layer 0's projection gradients take
// the token X = E + P as G^T dZ (G = the byte-embedding part, bf16 exact in
// Xk) plus P^T (sum over windows of dZ), later layers' their rounded input.
bool lower_backward(trace_model* m, int l, int64_t N64, hipStream_t s) {
  const Layout& L = m->L;
  const int T = L.T, D = L.D, F = m->cfg.F, H = m->cfg.H, k = m->cfg.k, N = (int)N64;
  const int rb = m->bf ? 1 : 0, hf = m->bf ? 1 : 0;
  const int R = N * T;
  const float* th = m->theta;
  float* gr = m->grad;
  float* ws = m->gws;
  const int64_t cap = m->gws_cap;
  const LowerKeep kp = lower_keep(m, l);
  const float* X = m->klX + (int64_t)l * m->max_keep * T * D;
  float* dY = m->ldY;
  bool ok = true;
  (void)hipMemcpyAsync(dY, m->dX, (size_t)R * D * 4, hipMemcpyDeviceToDevice, s);
  for (int r = k - 1; r >= 0; --r) {
    const int64_t wr = m->cfg.untied_ffn ? (int64_t)r * D * F : 0;
    const float beta = (r == k - 1 || m->cfg.untied_ffn) ? 0.f : 1.f;
    const float* U = kp.U + r * kp.us;
    const float* Y = kp.Y + r * kp.ys;
    GemmArgs gd = gemm(R, F, D, dY, D, 1, rb, th + L.at(P_W2, l) + wr, 1, D, rb, m->ldU, F, 0.f);
    gd.gelu_u = U;
    ok = launch_gemm(gd, ws, cap, s) && ok;
    launch_gelu_fwd_round(U, m->ldG, (int64_t)R * F, rb, s);
    ok = launch_gemm(gemm(F, D, R, m->ldG, 1, F, rb, dY, D, 1, rb, gr + L.at(P_W2, l) + wr, D, beta), ws, cap, s) &&
         ok;
    ok = launch_gemm(gemm(D, F, R, Y, 1, D, rb, m->ldU, F, 1, rb, gr + L.at(P_W1, l) + wr, F, beta), ws, cap, s) && ok;
    ok = launch_gemm(gemm(R, D, F, m->ldU, F, 1, rb, th + L.at(P_W1, l) + wr, 1, F, rb, dY, D, 1.f), ws, cap, s) && ok;
  }
  // dY is now dY_0: dWo = O^T dY_0, dO = dY_0 Wo^T, attention over every row
  ok = launch_gemm(gemm(D, D, R, kp.O, 1, D, rb, dY, D, 1, rb, gr + L.at(P_WO, l), D, 0.f), ws, cap, s) && ok;
  ok = launch_gemm(gemm(R, D, D, dY, D, 1, rb, th + L.at(P_WO, l), 1, D, rb, m->ldO, D, 0.f), ws, cap, s) && ok;
  launch_attn_bwd_rows(m->ldO, kp.Q, kp.K, kp.V, kp.A, N, T, D, H, (float)(1.0 / std::sqrt((double)L.DH)), rb,
                       m->ldQ, m->dK, m->dV, s);
  const float* dZ[3] = {m->ldQ, m->dK, m->dV};
  const int pz[3] = {P_WQ, P_WK, P_WV};
  for (int i = 0; i < 3; ++i) {
    if (l == 0) {
      GemmArgs g = gemm(D, D, R, m->Xk, 1, D, rb, dZ[i], D, 1, 0, gr + L.at(pz[i], l), D, 0.f);
      g.halfA = hf;
      ok = launch_gemm(g, ws, cap, s) && ok;
      if (m->cfg.use_pos) {
        launch_colsum(dZ[i], N, (int64_t)T * D, (int64_t)T * D, m->sP, 0.f, m->cws, s);
        launch_pos_grad(m->bf, m->Pc, m->sP, 0, T, D, gr + L.at(pz[i], l), s);
      }
    } else {
      ok = launch_gemm(gemm(D, D, R, X, 1, D, rb, dZ[i], D, 1, 0, gr + L.at(pz[i], l), D, 0.f), ws, cap, s) && ok;
    }
  }
  // dX = dQ Wq^T + dK Wk^T + dV Wv^T + dY_0
  launch_gemm2(gemm(R, D, D, m->dK, D, 1, 0, th + L.at(P_WK, l), 1, D, rb, m->dX, D, 0.f),
               gemm(R, D, D, m->dV, D, 1, 0, th + L.at(P_WV, l), 1, D, rb, m->dX, D, 0.f), ws, cap, s);
  ok = launch_gemm(gemm(R, D, D, m->ldQ, D, 1, 0, th + L.at(P_WQ, l), 1, D, rb, m->dX, D, 1.f), ws, cap, s) && ok;
  launch_add(m->dX, dY, R, D, D, D, s);
  return ok;
}

}  // namespace

extern "C" int trace_create(const trace_config* cfg, trace_model** out) {
  if (!out) return fail(TRACE_EINVAL, "out is NULL");
  *out = nullptr;
  Layout L;
  int rc = trace_check_config(cfg, &L);
  if (rc) return rc;
  const bool bf = cfg->dtype == TRACE_BF16;
  if (cfg->e % 8 != 0 || cfg->e > 128) return fail(TRACE_EUNSUPPORTED, "e must be a multiple of 8, at most 128");
  if (cfg->F % 256 != 0) return fail(TRACE_EUNSUPPORTED, "F must be a multiple of 256");
  if (cfg->g > 64 || cfg->W > 64) return fail(TRACE_EUNSUPPORTED, "W must be at most 64 bytes");
  if (cfg->max_keep * (int64_t)cfg->W >= ((int64_t)1 << 31))
    return fail(TRACE_EUNSUPPORTED, "max_keep * W must be below 2^31");
  attn_fn af = find_attn(bf, L.T, L.D, L.DH);
  ffn_fn ff = find_ffn(bf, L.D);
  if (!af || !ff)
    return fail(TRACE_EUNSUPPORTED, "no kernel for T=" + std::to_string(L.T) + " d=" + std::to_string(L.D) +
                                        " head width " + std::to_string(L.DH) + (bf ? " bf16" : " fp32"));
  trace_model* m = new (std::nothrow) trace_model();
  if (!m) return fail(TRACE_ENOMEM, "host allocation failed");
  m->cfg = *cfg;
  m->L = L;
  m->bf = bf;
  m->attn = af;
  m->ffn = ff;
  m->max_keep = cfg->max_keep;
  m->max_windows = std::max<int64_t>(std::max<int64_t>(cfg->max_windows, cfg->max_keep), 1);
  (void)hipGetDevice(&m->device);
  if (cfg->attention == TRACE_ATTN_PERFORMER)
    m->nfeat = cfg->n_features ? cfg->n_features : (L.DH <= 32 ? 128 : 256);
  const int64_t n = L.n, D = L.D, T = L.T, F = cfg->F, W = cfg->W;
  const int es = bf ? 2 : 4;
  bool ok = dalloc(m, &m->theta, n * 4) && dalloc(m, &m->am, n * 4) && dalloc(m, &m->av, n * 4) &&
            dalloc(m, &m->grad, n * 4) && dalloc(m, &m->Ec, L.size[P_E] * es) && dalloc(m, &m->Pc, L.size[P_P] * es) &&
            dalloc(m, &m->PW, 3 * T * D * 4) &&
            dalloc(m, &m->Wq, D * D * es) && dalloc(m, &m->Wk, D * D * es) && dalloc(m, &m->Wv, D * D * es) &&
            dalloc(m, &m->Wo, D * D * es) && dalloc(m, &m->W1, D * F * es * (cfg->untied_ffn ? cfg->k : 1)) &&
            dalloc(m, &m->W2, F * D * es * (cfg->untied_ffn ? cfg->k : 1)) &&
            dalloc(m, &m->Wout, D * 256 * es) && dalloc(m, &m->h0, m->max_windows * D * 4) &&
            (m->nfeat == 0 || dalloc(m, &m->Om, (int64_t)m->nfeat * L.DH * es));
  const int NL = L.NL, H = cfg->H, kk = cfg->k;
  if (ok && NL > 1) {
    // windows per forward chunk: the lower layers hold about T (7 D + 2 F)
    // floats per window
    m->lcap = std::max<int64_t>(std::min<int64_t>(m->max_windows, 16384), cfg->max_keep);
    const int64_t R = m->lcap * T;  // token rows
    m->fws_cap = 0;
    for (int64_t kd : {D, F})
      for (int64_t nd : {D, F})
        m->fws_cap = std::max(m->fws_cap, std::max(gemm_ws_floats((int)R, (int)nd, (int)kd),
                                                   bgemm_ws_floats((int)R, (int)nd, (int)kd)));
    ok = dalloc(m, &m->lx[0], R * D * 4) && dalloc(m, &m->lx[1], R * D * 4) && dalloc(m, &m->lq, R * D * 4) &&
         dalloc(m, &m->lk, R * D * 4) && dalloc(m, &m->lv, R * D * 4) && dalloc(m, &m->lo, R * D * 4) &&
         dalloc(m, &m->ly[0], R * D * 4) && dalloc(m, &m->ly[1], R * D * 4) && dalloc(m, &m->lu, R * F * 4) &&
         dalloc(m, &m->lg, R * F * 4) && dalloc(m, &m->fws, m->fws_cap * 4);
  }
  const int64_t K = cfg->max_keep;
  if (ok && K > 0 && NL > 1) {
    const int64_t R = K * T, nl = NL - 1;
    ok = dalloc(m, &m->klX, NL * R * D * 4) && dalloc(m, &m->klQ, nl * R * D * 4) &&
         dalloc(m, &m->klK, nl * R * D * 4) && dalloc(m, &m->klV, nl * R * D * 4) &&
         dalloc(m, &m->klA, nl * K * H * T * T * 4) && dalloc(m, &m->klO, nl * R * D * 4) &&
         dalloc(m, &m->klY, nl * kk * R * D * 4) && dalloc(m, &m->klU, nl * kk * R * F * 4) &&
         dalloc(m, &m->ldY, R * D * 4) && dalloc(m, &m->ldU, R * F * 4) && dalloc(m, &m->ldG, R * F * 4) &&
         dalloc(m, &m->ldO, R * D * 4) && dalloc(m, &m->ldQ, R * D * 4);
  }
  if (ok && K > 0) {
    ok = dalloc(m, &m->kwin, K * W) && dalloc(m, &m->ktgt, K * 4) && dalloc(m, &m->kq, K * D * 4) &&
         dalloc(m, &m->kK, K * T * D * 4) && dalloc(m, &m->kV, K * T * D * 4) &&
         dalloc(m, &m->kA, K * cfg->H * T * 4) && dalloc(m, &m->kO, K * D * 4) &&
         dalloc(m, &m->kY, (cfg->k + 1) * K * D * es) && dalloc(m, &m->kU, cfg->k * K * F * 4) &&
         (!bf || dalloc(m, &m->kG, cfg->k * K * F * 2)) &&
         dalloc(m, &m->kZ, K * 256 * 4) && dalloc(m, &m->dz, K * 256 * 4) &&
         dalloc(m, &m->dY, (cfg->k + 1) * K * D * 4) && dalloc(m, &m->dU, cfg->k * K * F * es) &&
         (bf || dalloc(m, &m->G, K * F * 4)) &&
         dalloc(m, &m->dO, K * D * 4) && dalloc(m, &m->dQ, K * D * 4) && dalloc(m, &m->dK, K * T * D * 4) &&
         dalloc(m, &m->dV, K * T * D * 4) && dalloc(m, &m->dX, K * T * D * 4) && dalloc(m, &m->Xk, K * T * D * es) &&
         dalloc(m, &m->sP, (2 * T + 2) * D * 4) &&
         dalloc(m, &m->apart, std::max(attn_bwd_part_floats(K, T, D, cfg->H), rank1_sums_part_floats(K, T, D)) * 4) &&
         dalloc(m, &m->dSc, K * cfg->H * T * 4) &&
         (!bf || (dalloc(m, &m->WkT, (int64_t)D * D * 2) && dalloc(m, &m->WvT, (int64_t)D * D * 2) &&
                  dalloc(m, &m->Wh, (m->L.off[P_BOUT] - m->L.off[P_WQ]) * 2))) &&
         dalloc(m, &m->gws, (m->gws_cap = adapt_gemm_ws(m, K)) * 4) &&
         dalloc(m, &m->ews, embed_bwd_ws_floats(K * W, cfg->e) * 4) &&
         dalloc(m, &m->cws, colsum_ws_floats(std::max<int64_t>((int64_t)(2 * T + 2) * D, 256)) * 4) &&
         dalloc(m, &m->gws2, m->gws_cap * 4) && dalloc(m, &m->cws2, colsum_ws_floats(T * D) * 4);
    if (ok) ok = hipStreamCreateWithFlags(&m->side, hipStreamNonBlocking) == hipSuccess;
    for (int i = 0; ok && i < 16; ++i) {
      hipEvent_t ev;
      ok = hipEventCreateWithFlags(&ev, hipEventDisableTiming) == hipSuccess;
      if (ok) m->sev.push_back(ev);
    }
  }
  if (!ok) {
    free_all(m);
    delete m;
    return fail(TRACE_ENOMEM, "device allocation failed");
  }
  hipError_t e = hipMemset(m->theta, 0, n * 4);
  if (e == hipSuccess) e = hipMemset(m->am, 0, n * 4);
  if (e == hipSuccess) e = hipMemset(m->av, 0, n * 4);
  if (e == hipSuccess) e = hipMemset(m->grad, 0, n * 4);
  if (e == hipSuccess && !refresh_operands(m, nullptr)) {
    free_all(m);
    delete m;
    return fail(TRACE_EUNSUPPORTED, "no operand refresh for this shape");
  }
  if (e == hipSuccess) e = hipDeviceSynchronize();
  if (e != hipSuccess) {
    rc = hip_fail(e, "trace_create");
    free_all(m);
    delete m;
    return rc;
  }
  // the fixed workspace of trace_forward_bits_noalloc on this device (if this
  // fails, that entry point retries and reports the error; nothing else uses it)
  (void)trace_scratch_setup(m->device);
  *out = m;
  return TRACE_OK;
}

extern "C" void trace_destroy(trace_model* m) {
  if (!m) return;
  (void)hipDeviceSynchronize();
  free_all(m);
  delete m;
}

extern "C" int trace_init_weights(trace_model* m, uint64_t seed, double stdv, const float* host_flat) {
  if (!m) return fail(TRACE_EINVAL, "model is NULL");
  if (!std::isfinite(stdv)) return fail(TRACE_EINVAL, "std must be finite");
  std::vector<float> h;
  const float* src = host_flat;
  if (!src) {
    h.resize((size_t)m->L.n);
    trace_fill_init(m->L, seed, stdv, h.data());
    src = h.data();
  }
  hipError_t e = hipMemcpy(m->theta, src, (size_t)m->L.n * 4, hipMemcpyHostToDevice);
  if (e == hipSuccess) e = hipMemset(m->am, 0, (size_t)m->L.n * 4);
  if (e == hipSuccess) e = hipMemset(m->av, 0, (size_t)m->L.n * 4);
  if (e != hipSuccess) return hip_fail(e, "trace_init_weights");
  m->step = 0;
  m->kept = false;
  refresh_operands(m, nullptr);
  e = hipDeviceSynchronize();
  if (e != hipSuccess) return hip_fail(e, "trace_init_weights");
  return TRACE_OK;
}

static int check_windows(const trace_model* m, const uint8_t* d_streams, int64_t stride, int32_t n_streams,
                         int64_t pos0, int32_t n_steps) {
  if (!m) return fail(TRACE_EINVAL, "model is NULL");
  if (!d_streams) return fail(TRACE_EINVAL, "streams is NULL");
  if (n_streams < 0 || n_steps < 0) return fail(TRACE_EINVAL, "n_streams and n_steps must be non-negative");
  if (pos0 < m->cfg.W) return fail(TRACE_EINVAL, "pos0 must be at least W (the first W bytes have no window)");
  if (n_streams > 1 && stride < pos0 + n_steps)
    return fail(TRACE_EINVAL, "stride shorter than the bytes each stream must hold (pos0 + n_steps)");
  return TRACE_OK;
}

namespace {
// fp32 -> bf16 bits, round to nearest even (finite inputs)
uint16_t host_bf16(float f) {
  uint32_t u;
  std::memcpy(&u, &f, 4);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}
}  // namespace

extern "C" int trace_set_features(trace_model* m, const float* omega, int64_t n) {
  if (!m || !omega) return fail(TRACE_EINVAL, "model or omega is NULL");
  if (m->cfg.attention != TRACE_ATTN_PERFORMER) return fail(TRACE_EINVAL, "the model does not use Performer attention");
  const int DH = m->L.DH, nf = m->nfeat;
  if (n != (int64_t)nf * DH) return fail(TRACE_EINVAL, "n must be n_features * d/H");
  for (int64_t i = 0; i < n; ++i)
    if (!std::isfinite(omega[i])) return fail(TRACE_EINVAL, "omega must be finite");
  // MFMA A fragments of omega, one per (16-feature block, k-step over the head
  // width), 64 lanes each, lane l holding feature 16 b + l % 16.  fp32: the
  // four k values 16 s + 4 (l/16) + t.  bf16: eight k values in the order in
  // which a lane holds the projected vector (two accumulator quads of 4
  // columns): j < 4 -> 32 s + 4 (l/16) + j, j >= 4 -> 32 s + 16 + 4 (l/16) + j - 4.
  const int kst = m->bf ? DH / 32 : DH / 16;
  std::vector<uint16_t> hb;
  std::vector<float> hf;
  if (m->bf)
    hb.resize((size_t)n);
  else
    hf.resize((size_t)n);
  for (int b = 0; b < nf / 16; ++b)
    for (int st = 0; st < kst; ++st)
      for (int l = 0; l < 64; ++l) {
        const int i = 16 * b + l % 16, lg = l / 16;
        const size_t base = ((size_t)(b * kst + st) * 64 + l);
        if (m->bf) {
          for (int j = 0; j < 8; ++j) {
            const int c = 32 * st + (j < 4 ? 4 * lg + j : 16 + 4 * lg + (j - 4));
            hb[base * 8 + j] = host_bf16(omega[(int64_t)i * DH + c]);
          }
        } else {
          for (int t = 0; t < 4; ++t) hf[base * 4 + t] = omega[(int64_t)i * DH + 16 * st + 4 * lg + t];
        }
      }
  hipError_t e = hipDeviceSynchronize();
  if (e == hipSuccess)
    e = hipMemcpy(m->Om, m->bf ? (const void*)hb.data() : (const void*)hf.data(), (size_t)n * (m->bf ? 2 : 4),
                  hipMemcpyHostToDevice);
  if (e != hipSuccess) return hip_fail(e, "trace_set_features");
  m->feats_set = true;
  return TRACE_OK;
}

int trace_model_dim(const trace_model* m) { return m->L.D; }
int trace_model_device(const trace_model* m) { return m->device; }

int trace_forward_into(trace_model* m, const uint8_t* d_streams, int64_t stride, int32_t n_streams, int64_t pos0,
                       int32_t n_steps, float* d_bits, float* d_logits, double* d_step_ce, uint32_t flags,
                       void* stream, float* h0, int64_t chunk_cap, bool timed) {
  int rc = check_windows(m, d_streams, stride, n_streams, pos0, n_steps);
  if (rc) return rc;
  if (flags & ~(uint32_t)(TRACE_KEEP_ACTS | TRACE_TOKEN_ATTN)) return fail(TRACE_EINVAL, "unknown flag");
  const bool keep = (flags & TRACE_KEEP_ACTS) != 0;
  const int64_t total = (int64_t)n_streams * n_steps;
  if (keep && (m->max_keep <= 0 || total > m->max_keep))
    return fail(TRACE_EINVAL, "KEEP_ACTS needs n_streams*n_steps <= max_keep");
  if (keep && total > chunk_cap) return fail(TRACE_EINVAL, "KEEP_ACTS batch larger than the workspace");
  if (total == 0) return TRACE_OK;  // nothing to write: output pointers may be NULL
  if (!d_bits) return fail(TRACE_EINVAL, "bits is NULL");
  if (m->nfeat && !m->feats_set) return fail(TRACE_ESTATE, "Performer features not set (trace_set_features)");
  const hipStream_t s = S(stream);
  const Layout& L = m->L;
  const int64_t chunk = keep ? total : (L.NL > 1 ? std::min(chunk_cap, m->lcap) : chunk_cap);
  const bool was_timing = m->timing;
  if (!timed) m->timing = false;
  bool lok = true;
  for (int64_t n0 = 0; n0 < total; n0 += chunk) {
    WinArgs w;
    w.streams = d_streams;
    w.stride = stride;
    w.pos0 = pos0;
    w.n_steps = n_steps;
    w.n0 = n0;
    w.N = std::min(chunk, total - n0);
    AttnArgs a;
    std::memset(&a, 0, sizeof(a));
    a.w = w;
    a.E = m->Ec;
    a.P = m->Pc;
    a.PW = m->PW;
    a.e = m->cfg.e;
    a.g = m->cfg.g;
    a.Wq = m->Wq;
    a.Wk = m->Wk;
    a.Wv = m->Wv;
    a.Wo = m->Wo;
    a.h0 = h0;
    a.token_only = (flags & TRACE_TOKEN_ATTN) != 0 || m->nfeat != 0 || L.NL > 1;
    if (L.NL > 1) {  // the lower layers over every token row; the top reads their output
      const int64_t R = w.N * L.T;
      float* X = keep ? m->klX : m->lx[0];
      launch_tokens(m->bf, w, m->Ec, m->Pc, L.T, L.D, m->cfg.e, m->cfg.g, X, s);
      for (int l = 0; l + 1 < L.NL; ++l) {
        LowerKeep kp;
        if (keep) kp = lower_keep(m, l);
        float* Xn = keep ? m->klX + (int64_t)(l + 1) * m->max_keep * L.T * L.D : m->lx[(l + 1) & 1];
        lok = lower_forward(m, l, X, Xn, w.N, keep ? &kp : nullptr, s) && lok;
        X = Xn;
        (void)R;
      }
      a.Xin = X;
    }
    a.Om = m->nfeat ? m->Om : nullptr;
    a.nfeat = m->nfeat;
    a.scale = (float)(1.0 / std::sqrt((double)L.DH));
    a.scale4 = (float)std::pow((double)L.DH, -0.25);
    FfnArgs f;
    std::memset(&f, 0, sizeof(f));
    f.w = w;
    f.h0 = h0;
    f.W1 = m->W1;
    f.W2 = m->W2;
    f.wstride = m->cfg.untied_ffn ? (int64_t)m->L.D * m->cfg.F * (m->bf ? 2 : 4) / 16 : 0;
    f.Wout = m->Wout;
    f.bout = m->theta + L.off[P_BOUT];
    f.F = m->cfg.F;
    f.k = m->cfg.k;
    f.bits = d_bits;
    f.logits = d_logits;
    if (keep) {
      a.kwin = m->kwin;
      a.kq = m->kq;
      a.kK = m->kK;
      a.kV = m->kV;
      a.kA = m->kA;
      a.kO = m->kO;
      f.kY = m->kY;
      f.kU = m->kU;
      f.kG = m->kG;
      f.kZ = m->kZ;
      f.ktgt = m->ktgt;
    }
    long tk = tbegin(m, s);
    m->attn(a, s);
    tend(m, tk, TRACE_KIND_ATTN, s);
    tk = tbegin(m, s);
    m->ffn(f, s);
    tend(m, tk, TRACE_KIND_FFN_HEAD, s);
  }
  if (d_step_ce && n_streams > 0) {
    const long tk = tbegin(m, s);
    launch_step_ce(d_bits, n_streams, n_steps, d_step_ce, s);
    tend(m, tk, TRACE_KIND_STEP_CE, s);
  }
  m->timing = was_timing;
  if (!lok) return fail(TRACE_EUNSUPPORTED, "a lower layer's product does not fit the GEMM kernels");
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_fail(e, "trace_forward_bits");
  if (keep) {
    m->kept = true;
    m->keepN = total;
  }
  return TRACE_OK;
}

extern "C" int trace_forward_bits(trace_model* m, const uint8_t* d_streams, int64_t stride, int32_t n_streams,
                                  int64_t pos0, int32_t n_steps, float* d_bits, float* d_logits, double* d_step_ce,
                                  uint32_t flags, void* stream) {
  if (!m) return fail(TRACE_EINVAL, "model is NULL");
  return trace_forward_into(m, d_streams, stride, n_streams, pos0, n_steps, d_bits, d_logits, d_step_ce, flags,
                            stream, m->h0, m->max_windows, true);
}

extern "C" int trace_adapt_step(trace_model* m, void* stream) {
  if (!m) return fail(TRACE_EINVAL, "model is NULL");
  if (m->nfeat) return fail(TRACE_EUNSUPPORTED, "the update covers softmax attention only (Performer: forward only)");
  if (!m->kept) return fail(TRACE_ESTATE, "no batch kept: run trace_forward_bits with TRACE_KEEP_ACTS first");
  const hipStream_t s = S(stream);
  const Layout& L = m->L;
  const int N = (int)m->keepN, D = L.D, T = L.T, F = m->cfg.F, H = m->cfg.H, k = m->cfg.k;
  const int rb = m->bf ? 1 : 0;  // bf16 storage points round their operands
  float* th = m->theta;
  float* gr = m->grad;
  float* ws = m->gws;
  const long tk = tbegin(m, s);
  bool ok = true;  // false if a product could not be launched
  // Two streams: s carries the chain of input gradients (dY, dU, dO, dQ/dK/dV,
  // dX, dE) and never waits for the other until the end; `side` computes the
  // weight gradients from the per-repeat buffers that chain leaves behind, each
  // as soon as its operands exist (a wait across streams costs several
  // microseconds, so only the side stream waits).  The side stream has its own
  // split-K and column-sum workspaces of the same sizes, so every product is the
  // same as on one stream.
  // Buffers by writer -> readers (every cross-stream read follows a mark of the
  // writer's stream, or, for the side stream's results, the final wait of s):
  //   s: dz -> s, side; dY_r, dU_r -> s, side (one buffer per repeat); dO, dX,
  //      grad P, grad E -> s; dQ, dK, dV -> s, side
  //   s: sums over windows in sP (dK, dV, dQ before the mark that the side
  //      stream waits on; dY_0 after it, read by s only)
  //   side: Xk, grad Wout, bout, W1, W2, Wo, Wq, Wk, Wv -> side only
  //   kept activations (forward, on s) -> both; s waits for side before Adam,
  //   so the next forward cannot overwrite them while side still reads
  const hipStream_t w = m->side;
  float* ws2 = m->gws2;
  auto dYr = [&](int r) { return m->dY + (int64_t)r * N * D; };  // w.r.t. the input of repeat r (r = k: Y_k)
  const int hf = m->bf ? 1 : 0;  // dU, Xk, kY stored as bf16
  // bf16 element e of a buffer whose elements are bf16 (hf) or fp32
  auto at = [&](float* p, int64_t e) { return hf ? (float*)((uint16_t*)p + e) : p + e; };
  auto dUr = [&](int r) { return at(m->dU, (int64_t)r * N * F); };
  // B operand from a weight of the master at offset o (Wq .. Wout): its bf16
  // image when the model keeps one (the same rounded values, half the bytes)
  const int hw = m->Wh ? 1 : 0;
  auto wsrc = [&](int64_t o) {
    return hw ? (const float*)(m->Wh + (o - L.off[P_WQ])) : (const float*)(th + o);
  };
  // stacked layers: this sequence runs the top layer (its weights at layer
  // NL - 1, its input the kept output of the layers below), then
  // lower_backward runs each lower layer down to the tokens
  const int NL = L.NL, top = NL - 1;
  const float* Xtop = NL > 1 ? m->klX + (int64_t)top * m->max_keep * T * D : nullptr;
  // head: dz = (softmax(z) - onehot) / N
  launch_ce_grad(m->kZ, m->ktgt, N, m->dz, s);
  order(m, s, w);
  // bf16 models: the key and value gradients are used through their rank-one
  // rows dK_h[n][t] = dS[n][h][t] scale q_h[n], dV_h[n][t] = A[n][h][t] bf(dO_h[n])
  // (the weight gradients from sums over each window's tokens, the input
  // gradient of the tokens by k_dx_rank1): dK, dV are not stored
  const bool pow2 = (T & (T - 1)) == 0 && (L.DH & (L.DH - 1)) == 0;
  const bool rank1 = m->bf && m->WkT && pow2 && dx_rank1_built(T, D, H);
  // one layer with those weight gradients: they gather their token rows
  // themselves, and only the last token's rows are gathered (dWq's operand)
  const bool kvfold = rank1 && NL == 1 && kv_wgrad_ready(N, T, D, H, m->cfg.e, m->gws_cap) &&
                      L.at(P_WV, top) == L.at(P_WK, top) + (int64_t)D * D;
  // side: the byte-embedding part of the tokens (read by the projection
  // gradients), dWout = h_k^T . dz and dbout = sum_n dz
  const bool xlast = kvfold && launch_gather_last(m->kwin, N, (const uint16_t*)m->Ec, T, D, m->cfg.e, m->cfg.g,
                                                 (uint16_t*)m->Xk, w);
  if (!xlast) launch_gather_kept(m->bf, m->kwin, N, m->Ec, T, D, m->cfg.e, m->cfg.g, m->Xk, w);
  GemmArgs go =
      gemm(D, 256, N, at(m->kY, (int64_t)k * N * D), 1, D, rb, m->dz, 256, 1, rb, gr + L.off[P_WOUT], 256, 0.f);
  go.halfA = hf;
  ok = launch_gemm(go, ws2, m->gws_cap, w) && ok;
  launch_colsum(m->dz, N, 256, 256, gr + L.off[P_BOUT], 0.f, m->cws2, w);
  // dY_k = dz . Wout^T
  GemmArgs gk = gemm(N, D, 256, m->dz, 256, 1, rb, wsrc(L.off[P_WOUT]), 1, 256, rb, dYr(k), D, 0.f);
  gk.halfB = hw;
  ok = launch_gemm(gk, ws, m->gws_cap, s) && ok;
  // shared FFN, repeats in reverse: dU_r = (dY_{r+1} . W2^T) * GELU'(U_r),
  // dY_r = dY_{r+1} + dU_r . W1^T; once dU_r exists the side stream forms
  // dW2 += G_r^T . dY_{r+1} and dW1 += Y_r^T . dU_r (accumulated over the repeats
  // in reverse; G = GELU(U) at its storage point: kept by the bf16 forward,
  // formed here otherwise).  With shared weights and G kept, the sums over the
  // repeats are single products over k N rows instead (the per-repeat buffers
  // are consecutive: G_0..G_{k-1} with dY_1..dY_k, Y_0..Y_{k-1} with dU_0..dU_{k-1}),
  // formed on the side stream once dO is done (below).
  const bool merged = m->kG && !m->cfg.untied_ffn;
  for (int r = k - 1; r >= 0; --r) {
    // untied FFN: repeat r's own W1, W2 and gradient blocks (each written once)
    const int64_t wr = m->cfg.untied_ffn ? (int64_t)r * D * F : 0;
    GemmArgs gd = gemm(N, F, D, dYr(r + 1), D, 1, rb, wsrc(L.at(P_W2, top) + wr), 1, D, rb, dUr(r), F, 0.f);
    gd.gelu_u = m->kU + (int64_t)r * N * F;
    gd.halfC = hf;
    gd.halfB = hw;
    ok = launch_gemm(gd, ws, m->gws_cap, s) && ok;
    if (!merged) {
      order(m, s, w);  // dY_{r+1} and dU_r are complete
      const float beta = (r == k - 1 || m->cfg.untied_ffn) ? 0.f : 1.f;
      GemmArgs g2w;
      if (m->kG) {
        g2w = gemm(F, D, N, (const float*)(m->kG + (int64_t)r * N * F), 1, F, rb, dYr(r + 1), D, 1, rb,
                   gr + L.at(P_W2, top) + wr, D, beta);
        g2w.halfA = 1;
      } else {
        launch_gelu_fwd_round(m->kU + (int64_t)r * N * F, m->G, (int64_t)N * F, rb, w);
        g2w = gemm(F, D, N, m->G, 1, F, rb, dYr(r + 1), D, 1, rb, gr + L.at(P_W2, top) + wr, D, beta);
      }
      ok = launch_gemm(g2w, ws2, m->gws_cap, w) && ok;
      GemmArgs g1w =
          gemm(D, F, N, at(m->kY, (int64_t)r * N * D), 1, D, rb, dUr(r), F, 1, rb, gr + L.at(P_W1, top) + wr, F, beta);
      g1w.halfA = g1w.halfB = hf;
      ok = launch_gemm(g1w, ws2, m->gws_cap, w) && ok;
    }
    // dY_r = dY_{r+1} + dU_r . W1^T (the addend read from dY_{r+1}'s own buffer)
    GemmArgs gy = gemm(N, D, F, dUr(r), F, 1, rb, wsrc(L.at(P_W1, top) + wr), 1, F, rb, dYr(r), D, 1.f);
    gy.Cin = dYr(r + 1);
    gy.halfA = hf;
    gy.halfB = hw;
    ok = launch_gemm(gy, ws, m->gws_cap, s) && ok;
  }
  // attention output projection: dO = dY_0 . Wo^T, then the attention (last
  // query row) -> dQ, dK, dV
  GemmArgs go2 = gemm(N, D, D, dYr(0), D, 1, rb, wsrc(L.at(P_WO, top)), 1, D, rb, m->dO, D, 0.f);
  go2.halfB = hw;
  ok = launch_gemm(go2, ws, m->gws_cap, s) && ok;
  // the side stream's large products start once dO is done (dY_0 complete), so
  // that they share the CUs with the attention backward's memory-bound kernels
  // rather than with the FFN chain's products
  order(m, s, w);
  if (merged) {
    // dW2 = sum_r G_r^T dY_{r+1} and dW1 = sum_r Y_r^T dU_r over the k N rows
    GemmArgs g2w = gemm(F, D, k * N, (const float*)m->kG, 1, F, rb, dYr(1), D, 1, rb, gr + L.at(P_W2, top), D, 0.f);
    g2w.halfA = 1;
    ok = launch_gemm(g2w, ws2, m->gws_cap, w) && ok;
    GemmArgs g1w = gemm(D, F, k * N, m->kY, 1, D, rb, m->dU, F, 1, rb, gr + L.at(P_W1, top), F, 0.f);
    g1w.halfA = g1w.halfB = hf;
    ok = launch_gemm(g1w, ws2, m->gws_cap, w) && ok;
  }
  // side: dWo = O^T . dY_0
  launch_gemm(gemm(D, D, N, m->kO, 1, D, rb, dYr(0), D, 1, rb, gr + L.at(P_WO, top), D, 0.f), ws2, m->gws_cap, w);
  // sP: [0, T D) sum over windows of dK, [T D, 2T D) of dV (from the attention
  // backward), [2T D, (2T+1) D) of dQ, [(2T+1) D, (2T+2) D) of dY_0
  float* sK = m->sP;
  float* sV = m->sP + (int64_t)T * D;
  float* sQ = m->sP + (int64_t)2 * T * D;
  float* sY = m->sP + (int64_t)(2 * T + 1) * D;
  const float ascale = (float)(1.0 / std::sqrt((double)L.DH));
  // rank1: the sums over windows of dK and dV (sK, sV; read by the positional
  // gradients of a single layer only) from the rank-one rows, with those of dQ
  // and dY_0 (sQ, sY) in the same pass
  const bool sums1 = rank1 && NL == 1 && m->cfg.use_pos;
  launch_attn_bwd(m->dO, m->kq, m->kK, m->kV, m->kA, N, T, D, H, ascale, rb, m->dQ, rank1 ? nullptr : m->dK,
                  rank1 ? nullptr : m->dV, rank1 ? nullptr : m->apart, sK, m->cws, s, m->bf ? m->dSc : nullptr);
  if (sums1 &&
      !launch_rank1_sums(m->dSc, m->kq, m->kA, m->dO, m->dQ, dYr(0), N, T, D, H, ascale, rb, m->apart, sK, m->cws, s))
    ok = false;
  auto log2i = [](int x) {
    int r = 0;
    while ((1 << r) < x) ++r;
    return r;
  };
  // B of X^T dK (rank1: from dS and q) and of X^T dV (rank1: from A and bf(dO))
  auto kv_grad = [&](const float* Aop, int64_t sam, int64_t sak, bool halfA, bool value, float* C) {
    GemmArgs g = rank1 ? gemm(D, D, N * T, Aop, sam, sak, rb, value ? m->dO : m->kq, D, 1, 0, C, D, 0.f)
                       : gemm(D, D, N * T, Aop, sam, sak, rb, value ? m->dV : m->dK, D, 1, 0, C, D, 0.f);
    g.halfA = halfA ? 1 : 0;
    if (rank1) {
      g.r1c = value ? m->kA : m->dSc;
      g.r1tsh = log2i(T);
      g.r1dsh = log2i(L.DH);
      g.r1H = H;
      g.r1round = value ? rb : 0;
      g.r1scale = value ? 1.f : ascale;
    }
    return launch_gemm(g, ws2, m->gws_cap, w);
  };
  if (m->cfg.use_pos && !sums1) launch_colsum(m->dQ, N, D, D, sQ, 0.f, m->cws, s);
  order(m, s, w);  // dQ, dK, dV and their sums over windows are complete
  // side: dWk = X^T dK, dWv = X^T dV (dK, dV stay fp32), with X = G + P[t]:
  // G^T dZ as GEMMs on the byte-embedding part G, then P^T (sum over windows of
  // dZ) for the positional part
  if (NL == 1) {
    // rank1: both from the per-window sums over the tokens (one launch; xlast:
    // their rows gathered in it, Xk holding the last tokens only)
    if (xlast) {
      ok = launch_kv_wgrad(nullptr, m->kwin, (const uint16_t*)m->Ec, m->cfg.e, m->cfg.g, m->dSc, m->kA, m->kq, m->dO,
                           N, T, D, H, ascale, ws2, m->gws_cap, gr + L.at(P_WK, top), gr + L.at(P_WV, top), w) &&
           ok;
    } else if (!(rank1 && launch_kv_wgrad((const uint16_t*)m->Xk, nullptr, nullptr, 8, 1, m->dSc, m->kA, m->kq,
                                          m->dO, N, T, D, H, ascale, ws2, m->gws_cap, gr + L.at(P_WK, top),
                                          gr + L.at(P_WV, top), w))) {
      ok = kv_grad(m->Xk, 1, D, hf, false, gr + L.at(P_WK, top)) && ok;
      ok = kv_grad(m->Xk, 1, D, hf, true, gr + L.at(P_WV, top)) && ok;
    }
    // side: dWq = X_last^T dQ; Xk was written on this stream, dQ before the last mark
    GemmArgs gq = xlast ? gemm(D, D, N, m->Xk, 1, D, rb, m->dQ, D, 1, 0, gr + L.at(P_WQ, top), D, 0.f)
                        : gemm(D, D, N, at(m->Xk, (int64_t)(T - 1) * D), 1, (int64_t)T * D, rb, m->dQ, D, 1, 0,
                               gr + L.at(P_WQ, top), D, 0.f);
    gq.halfA = hf;
    ok = launch_gemm(gq, ws2, m->gws_cap, w) && ok;
    if (m->cfg.use_pos) {
      // the positional parts of dWk, dWv, dWq in one launch
      const float* S3[3] = {sK, sV, sQ};
      const int t03[3] = {0, 0, T - 1}, nt3[3] = {T, T, 1};
      float* dW3[3] = {gr + L.at(P_WK, top), gr + L.at(P_WV, top), gr + L.at(P_WQ, top)};
      launch_pos_grad3(m->bf, m->Pc, S3, t03, nt3, dW3, 3, D, w);
    }
  } else {
    // the top layer's input: the layer below's output, rounded (bf16 storage point)
    ok = kv_grad(Xtop, 1, D, false, false, gr + L.at(P_WK, top)) && ok;
    ok = kv_grad(Xtop, 1, D, false, true, gr + L.at(P_WV, top)) && ok;
    ok = launch_gemm(gemm(D, D, N, Xtop + (int64_t)(T - 1) * D, 1, (int64_t)T * D, rb, m->dQ, D, 1, 0,
                          gr + L.at(P_WQ, top), D, 0.f),
                     ws2, m->gws_cap, w) && ok;
  }
  // dX = dK Wk^T + dV Wv^T (+ dQ Wq^T + dY_0 on the last token).  bf16 models
  // form the key and value part from the rank-one rows of dK and dV
  // (launch_dx_rank1, which adds dY_0); otherwise two products over every token
  // row, then dY_0
  if (rank1) ok = launch_dx_rank1(m->kq, m->dO, m->dSc, m->kA, m->WkT, m->WvT, dYr(0), N, T, D, H, ascale, m->dX, s) && ok;
  if (!rank1) {
    GemmArgs gxk = gemm(N * T, D, D, m->dK, D, 1, 0, wsrc(L.at(P_WK, top)), 1, D, rb, m->dX, D, 0.f);
    GemmArgs gxv = gemm(N * T, D, D, m->dV, D, 1, 0, wsrc(L.at(P_WV, top)), 1, D, rb, m->dX, D, 0.f);
    gxk.halfB = gxv.halfB = hw;
    launch_gemm2(gxk, gxv, ws, m->gws_cap, s);
  }
  GemmArgs gxq = gemm(N, D, D, m->dQ, D, 1, 0, wsrc(L.at(P_WQ, top)), 1, D, rb, m->dX + (int64_t)(T - 1) * D,
                      (int64_t)T * D, 1.f);
  gxq.halfB = hw;
  ok = launch_gemm(gxq, ws, m->gws_cap, s) && ok;
  if (!rank1) launch_add(m->dX + (int64_t)(T - 1) * D, dYr(0), N, D, (int64_t)T * D, D, s);
  if (NL > 1) {
    // dX is the gradient w.r.t. the top layer's input: down through the lower
    // layers (on this stream, after the side stream's work: layer 0 reads Xk)
    order(m, w, s);
    for (int l = NL - 2; l >= 0; --l) ok = lower_backward(m, l, N, s) && ok;
    if (m->cfg.use_pos)
      launch_colsum(m->dX, N, (int64_t)T * D, (int64_t)T * D, gr + L.off[P_P], 0.f, m->cws, s);
    else
      launch_zero(gr + L.off[P_P], L.size[P_P], s);
  } else if (m->cfg.use_pos) {
    // positional table: dP[t] = sum_n dX[n][t], from the sums over windows of
    // dK, dV, dQ and dY_0 times the weights; then the byte embedding
    if (!sums1) launch_colsum(dYr(0), N, D, D, sY, 0.f, m->cws, s);
    launch_pos_table_grad(sK, sQ, sY, th + L.at(P_WQ, top), th + L.at(P_WK, top), th + L.at(P_WV, top), T, D, rb,
                          gr + L.off[P_P], s);
  } else {
    launch_zero(gr + L.off[P_P], L.size[P_P], s);
  }
  launch_embed_bwd(m->kwin, m->dX, N, m->cfg.W, m->cfg.e, gr + L.off[P_E], m->ews, s);
  order(m, w, s);  // every gradient is complete
  if (!ok) {
    tend(m, tk, TRACE_KIND_BACKWARD, s);
    return fail(TRACE_EUNSUPPORTED, "trace_adapt_step: an operand stored as bf16 does not fit the bf16 GEMM");
  }
  tend(m, tk, TRACE_KIND_BACKWARD, s);
  // Adam on the flat master, then new operand copies
  m->step += 1;
  m->upd_run = true;
  const float bc1 = (float)(1.0 - std::pow(m->cfg.beta1, (double)m->step));
  const float bc2 = (float)(1.0 - std::pow(m->cfg.beta2, (double)m->step));
  // one kernel: its dispatch records the two events itself, so the region is the kernel's own duration
  const long ta = treserve(m);
  launch_adam(th, gr, m->am, m->av, L.n, (float)m->cfg.lr, (float)m->cfg.beta1, (float)m->cfg.beta2,
              (float)m->cfg.eps, bc1, bc2, s, ta >= 0 ? m->events[2 * ta] : nullptr,
              ta >= 0 ? m->events[2 * ta + 1] : nullptr);
  if (ta >= 0) m->ev_kind[ta] = TRACE_KIND_ADAM;
  refresh_operands(m, s);
  m->kept = false;
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_fail(e, "trace_adapt_step");
  return TRACE_OK;
}

extern "C" int trace_get_state(trace_model* m, float* theta, float* adam_m, float* adam_v, int64_t* step, int64_t n) {
  if (!m) return fail(TRACE_EINVAL, "model is NULL");
  if (n != m->L.n) return fail(TRACE_EINVAL, "n must equal trace_param_count");
  hipError_t e = hipDeviceSynchronize();
  if (e == hipSuccess && theta) e = hipMemcpy(theta, m->theta, n * 4, hipMemcpyDeviceToHost);
  if (e == hipSuccess && adam_m) e = hipMemcpy(adam_m, m->am, n * 4, hipMemcpyDeviceToHost);
  if (e == hipSuccess && adam_v) e = hipMemcpy(adam_v, m->av, n * 4, hipMemcpyDeviceToHost);
  if (e != hipSuccess) return hip_fail(e, "trace_get_state");
  if (step) *step = m->step;
  return TRACE_OK;
}

extern "C" int trace_set_state(trace_model* m, const float* theta, const float* adam_m, const float* adam_v,
                               int64_t step, int64_t n) {
  if (!m) return fail(TRACE_EINVAL, "model is NULL");
  if (n != m->L.n) return fail(TRACE_EINVAL, "n must equal trace_param_count");
  if (step < 0) return fail(TRACE_EINVAL, "step must be non-negative");
  hipError_t e = hipDeviceSynchronize();
  if (e == hipSuccess && theta) e = hipMemcpy(m->theta, theta, n * 4, hipMemcpyHostToDevice);
  if (e == hipSuccess && adam_m) e = hipMemcpy(m->am, adam_m, n * 4, hipMemcpyHostToDevice);
  if (e == hipSuccess && adam_v) e = hipMemcpy(m->av, adam_v, n * 4, hipMemcpyHostToDevice);
  if (e != hipSuccess) return hip_fail(e, "trace_set_state");
  m->step = step;
  m->kept = false;
  refresh_operands(m, nullptr);
  e = hipDeviceSynchronize();
  if (e != hipSuccess) return hip_fail(e, "trace_set_state");
  return TRACE_OK;
}

extern "C" int trace_get_grads(trace_model* m, float* host_out, int64_t n) {
  if (!m || !host_out) return fail(TRACE_EINVAL, "model or output is NULL");
  if (n != m->L.n) return fail(TRACE_EINVAL, "n must equal trace_param_count");
  hipError_t e = hipDeviceSynchronize();
  if (e == hipSuccess) e = hipMemcpy(host_out, m->grad, n * 4, hipMemcpyDeviceToHost);
  if (e != hipSuccess) return hip_fail(e, "trace_get_grads");
  return TRACE_OK;
}

extern "C" int trace_debug_kept_tokens(trace_model* m, void* d_X, void* stream) {
  if (!m || !d_X) return fail(TRACE_EINVAL, "model or X is NULL");
  if (!m->kept) return fail(TRACE_ESTATE, "no batch kept: run trace_forward_bits with TRACE_KEEP_ACTS first");
  // the update's own gather (trace_adapt_step), on the window bytes the
  // attention kernel kept
  launch_gather_kept(m->bf, m->kwin, m->keepN, m->Ec, m->L.T, m->L.D, m->cfg.e, m->cfg.g, d_X, S(stream));
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_fail(e, "trace_debug_kept_tokens");
  return TRACE_OK;
}

extern "C" int trace_debug_kv_wgrad(trace_model* m, float* d_gathered, float* d_rows, void* stream) {
  if (!m || !d_gathered || !d_rows) return fail(TRACE_EINVAL, "model or output is NULL");
  if (!m->upd_run) return fail(TRACE_ESTATE, "no update yet: run trace_adapt_step first");
  const Layout& L = m->L;
  const int64_t N = m->keepN;
  const int T = L.T, D = L.D, H = m->cfg.H;
  const bool pow2 = (T & (T - 1)) == 0 && (L.DH & (L.DH - 1)) == 0;
  if (!m->bf || !m->WkT || !pow2 || !dx_rank1_built(T, D, H) || L.NL != 1 ||
      !kv_wgrad_ready(N, T, D, H, m->cfg.e, m->gws_cap))
    return fail(TRACE_EUNSUPPORTED, "trace_debug_kv_wgrad: not a shape of the rank-one weight-gradient kernel");
  const hipStream_t s = S(stream);
  const float ascale = (float)(1.0 / std::sqrt((double)L.DH));
  const int64_t DD = (int64_t)D * D;
  launch_gather_kept(true, m->kwin, N, m->Ec, T, D, m->cfg.e, m->cfg.g, m->Xk, s);
  bool ok = launch_kv_wgrad((const uint16_t*)m->Xk, nullptr, nullptr, 8, 1, m->dSc, m->kA, m->kq, m->dO, N, T, D, H,
                            ascale, m->gws2, m->gws_cap, d_rows, d_rows + DD, s);
  ok = ok && launch_kv_wgrad(nullptr, m->kwin, (const uint16_t*)m->Ec, m->cfg.e, m->cfg.g, m->dSc, m->kA, m->kq, m->dO,
                             N, T, D, H, ascale, m->gws2, m->gws_cap, d_gathered, d_gathered + DD, s);
  if (!ok) return fail(TRACE_EUNSUPPORTED, "trace_debug_kv_wgrad: the kernel did not take the operands");
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_fail(e, "trace_debug_kv_wgrad");
  return TRACE_OK;
}

extern "C" int trace_debug_gemm(int M, int N, int K, const void* d_A, int a_kc, int mode_a, const void* d_B, int b_kc,
                                int mode_b, void* d_C, int half_c, int kernel, float* d_ws, int64_t ws_floats,
                                void* stream) {
  if (M <= 0 || N <= 0 || K <= 0) return fail(TRACE_EINVAL, "M, N, K must be positive");
  if (!d_A || !d_B || !d_C) return fail(TRACE_EINVAL, "A, B or C is NULL");
  if (mode_a < 0 || mode_a > 2 || mode_b < 0 || mode_b > 2 || (mode_a == 1 && mode_b == 1))
    return fail(TRACE_EINVAL, "modes are 0, 1, 2, and at most one operand is split");
  if (kernel != 1 && kernel != 2) return fail(TRACE_EINVAL, "kernel must be 1 or 2");
  if (ws_floats < 0 || (ws_floats > 0 && !d_ws)) return fail(TRACE_EINVAL, "workspace");
  GemmArgs g = gemm(M, N, K, (const float*)d_A, a_kc ? K : 1, a_kc ? 1 : M, mode_a != 1, (const float*)d_B,
                    b_kc ? 1 : N, b_kc ? K : 1, mode_b != 1, (float*)d_C, N, 0.f);
  g.halfA = mode_a == 2;
  g.halfB = mode_b == 2;
  g.halfC = half_c != 0;
  if (!launch_bgemm(g, nullptr, d_ws, ws_floats, S(stream), kernel))
    return fail(TRACE_EUNSUPPORTED, "trace_debug_gemm: the operands do not fit the bf16 kernel");
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_fail(e, "trace_debug_gemm");
  return TRACE_OK;
}

extern "C" int trace_set_timing(trace_model* m, int enable) {
  if (!m) return fail(TRACE_EINVAL, "model is NULL");
  m->timing = enable != 0;
  return TRACE_OK;
}

extern "C" int trace_read_timing(trace_model* m, double* ms_total, int64_t* launches, int64_t* overflow) {
  if (!m || !ms_total || !launches) return fail(TRACE_EINVAL, "model or output is NULL");
  for (int k = 0; k < TRACE_NKINDS; ++k) {
    ms_total[k] = 0.0;
    launches[k] = 0;
  }
  const int rc = harvest(m) ? TRACE_OK : fail(TRACE_EHIP, "trace_read_timing: an event could not be read");
  for (int k = 0; k < TRACE_NKINDS; ++k) {
    ms_total[k] = m->t_ms[k];
    launches[k] = m->t_n[k];
    m->t_ms[k] = 0.0;
    m->t_n[k] = 0;
  }
  if (overflow) *overflow = m->overflow;
  m->overflow = 0;
  return rc;
}

// ------------------------------------------------------------- coding ----
#include <condition_variable>
#include <functional>
#include <mutex>
#include <thread>

#include "codec.h"

namespace {
// Host threads kept for one compress or decompress call: run(n, fn) calls
// fn(b0, b1) over [0, n) in contiguous pieces, one per thread (one thread
// below 512 items, up to 16), and returns when all pieces are done.  Each item
// is written by one thread only.
class WorkPool {
 public:
  explicit WorkPool(int64_t n_items) {
    const int64_t hw = std::max<int64_t>(1, std::min<int64_t>(16, (int64_t)std::thread::hardware_concurrency()));
    nt_ = n_items < 512 ? 1 : std::min<int64_t>(hw, n_items / 256);
    for (int64_t t = 1; t < nt_; ++t) th_.emplace_back([this, t] { worker(t); });
  }
  ~WorkPool() {
    {
      std::lock_guard<std::mutex> lk(mu_);
      stop_ = true;
    }
    cv_.notify_all();
    for (auto& x : th_) x.join();
  }
  void run(int64_t n, const std::function<void(int64_t, int64_t)>& fn) {
    if (nt_ <= 1) {
      fn(0, n);
      return;
    }
    {
      std::lock_guard<std::mutex> lk(mu_);
      fn_ = &fn;
      n_ = n;
      left_ = nt_ - 1;
      ++gen_;
    }
    cv_.notify_all();
    fn(0, n / nt_);
    std::unique_lock<std::mutex> lk(mu_);
    done_.wait(lk, [&] { return left_ == 0; });
  }

 private:
  void worker(int64_t t) {
    int64_t seen = 0;
    for (;;) {
      const std::function<void(int64_t, int64_t)>* f;
      int64_t n;
      {
        std::unique_lock<std::mutex> lk(mu_);
        cv_.wait(lk, [&] { return stop_ || gen_ != seen; });
        if (stop_) return;
        seen = gen_;
        f = fn_;
        n = n_;
      }
      (*f)(n * t / nt_, n * (t + 1) / nt_);
      std::lock_guard<std::mutex> lk(mu_);
      if (--left_ == 0) done_.notify_one();
    }
  }
  int64_t nt_ = 1, n_ = 0, left_ = 0, gen_ = 0;
  bool stop_ = false;
  const std::function<void(int64_t, int64_t)>* fn_ = nullptr;
  std::vector<std::thread> th_;
  std::mutex mu_;
  std::condition_variable cv_, done_;
};
}  // namespace

extern "C" int trace_quant_table(uint32_t* out) {
  if (!out) return fail(TRACE_EINVAL, "out is NULL");
  std::memcpy(out, quant_table(), 256 * sizeof(uint32_t));
  return TRACE_OK;
}

extern "C" int trace_quantize(const float* d_logits, int64_t n, uint16_t* d_freq, void* stream) {
  if (n < 0) return fail(TRACE_EINVAL, "n must be non-negative");
  if (n > 0 && (!d_logits || !d_freq)) return fail(TRACE_EINVAL, "NULL buffer");
  if (((uintptr_t)d_logits & 15) || ((uintptr_t)d_freq & 7))
    return fail(TRACE_EINVAL, "logits must be 16-byte and freq 8-byte aligned");
  launch_quantize(d_logits, n, d_freq, (hipStream_t)stream);
  const hipError_t e = hipGetLastError();
  return e == hipSuccess ? TRACE_OK : hip_fail(e, "trace_quantize");
}

extern "C" int trace_rc_encode(const uint16_t* freq, int64_t freq_stride, const uint8_t* sym, int64_t n, uint8_t* out,
                               int64_t cap, int64_t* size) {
  if (n < 0 || cap < 0 || freq_stride < 0) return fail(TRACE_EINVAL, "negative size");
  if ((n > 0 && (!sym || (freq_stride > 0 && !freq))) || !size || (cap > 0 && !out))
    return fail(TRACE_EINVAL, "NULL buffer");
  RcEnc enc;
  enc.out = out;
  enc.cap = cap;
  for (int64_t i = 0; i < n; ++i) {
    const int x = sym[i];
    if (freq_stride == 0) {
      enc.encode((uint32_t)x, 1, 256);
      continue;
    }
    const uint16_t* f = freq + i * freq_stride;
    uint32_t cum = 0, tot = 0;
    for (int s = 0; s < 256; ++s) {
      if (s < x) cum += f[s];
      tot += f[s];
    }
    if (f[x] == 0 || tot > 65536) return fail(TRACE_EINVAL, "frequencies must be >= 1 with a total of at most 65536");
    enc.encode(cum, f[x], tot);
  }
  enc.finish();
  *size = enc.n;
  return enc.over() ? fail(TRACE_EINVAL, "out is too small for the code (size holds the length needed)") : TRACE_OK;
}

extern "C" int trace_rc_decode(const uint16_t* freq, int64_t freq_stride, const uint8_t* in, int64_t size, int64_t n,
                               uint8_t* sym_out) {
  if (n < 0 || size < 0 || freq_stride < 0) return fail(TRACE_EINVAL, "negative size");
  if ((n > 0 && (!sym_out || (freq_stride > 0 && !freq))) || (size > 0 && !in)) return fail(TRACE_EINVAL, "NULL buffer");
  RcDec dec;
  dec.in = in;
  dec.size = size;
  dec.start();
  for (int64_t i = 0; i < n; ++i) {
    if (freq_stride == 0) {
      sym_out[i] = (uint8_t)dec.decode_uniform();
      continue;
    }
    const uint16_t* f = freq + i * freq_stride;
    uint32_t tot = 0;
    for (int s = 0; s < 256; ++s) {
      if (f[s] == 0) return fail(TRACE_EINVAL, "frequencies must be >= 1");
      tot += f[s];
    }
    if (tot > 65536) return fail(TRACE_EINVAL, "frequency total above 65536");
    sym_out[i] = (uint8_t)dec.decode(f, 256, tot);
  }
  return TRACE_OK;
}

namespace {
// The loop of Alg. 1 shared by both directions over n_streams streams of
// `length` bytes: bytes [0, W) at 1/256 (lines 1-5); at each i >= W one
// forward over the windows ending before i (line 8) -> frequencies -> the
// coding step code(i, freq) (line 9, which leaves the bytes at i in h) -> the
// controller on the batch-mean coded length (Alg. 2) -> if it says so, the
// forward again keeping activations and the backward + Adam (line 10).
// d_src holds the bytes the forwards read; after code(i) its column i holds
// the bytes at i (the targets of the keeping forward).
template <class First, class Code>
int coding_loop(trace_model* m, const uint8_t* d_src, int64_t stride, int32_t B, int64_t length, int32_t mode,
                int32_t ctl_t, double ctl_delta, int64_t* n_updates, void* stream, First first, Code code) {
  const int W = m->cfg.W;
  hipStream_t s = (hipStream_t)stream;
  trace_controller ctl;
  if (mode == 1) {
    const int rc = trace_controller_init(&ctl, ctl_t, ctl_delta);
    if (rc) return rc;
  }
  int rc = first((int64_t)std::min<int64_t>(W, length));
  if (rc) return rc;
  if (length <= W) {
    if (n_updates) *n_updates = 0;
    return TRACE_OK;
  }
  float *d_logits = nullptr, *d_bits = nullptr;
  uint16_t* d_freq = nullptr;
  hipError_t e = hipMalloc(&d_logits, (size_t)B * 256 * 4);
  if (e == hipSuccess) e = hipMalloc(&d_bits, (size_t)B * 4);
  if (e == hipSuccess) e = hipMalloc(&d_freq, (size_t)B * 256 * 2);
  // frequencies land in pinned host memory (one direct copy per position)
  uint16_t* hf = nullptr;
  if (e == hipSuccess) e = hipHostMalloc((void**)&hf, (size_t)B * 256 * 2, hipHostMallocDefault);
  int64_t updates = 0;
  rc = e == hipSuccess ? TRACE_OK : hip_fail(e, "coding buffers");
  for (int64_t i = W; i < length && rc == TRACE_OK; ++i) {
    rc = trace_forward_bits(m, d_src, stride, B, i, 1, d_bits, d_logits, nullptr, 0, stream);
    if (rc) break;
    launch_quantize(d_logits, B, d_freq, s);
    e = hipMemcpyAsync(hf, d_freq, (size_t)B * 256 * 2, hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) {
      rc = hip_fail(e, "coding step");
      break;
    }
    double ce = 0.0;
    rc = code(i, hf, &ce);
    if (rc) break;
    ce /= B;
    int32_t upd = mode == 2 ? 1 : 0;
    if (mode == 1) {
      rc = trace_controller_decide(&ctl, ce, &upd);
      if (rc) break;
    }
    if (upd) {
      rc = trace_forward_bits(m, d_src, stride, B, i, 1, d_bits, nullptr, nullptr, TRACE_KEEP_ACTS, stream);
      if (!rc) rc = trace_adapt_step(m, stream);
      ++updates;
    }
  }
  hipFree(d_logits);
  hipFree(d_bits);
  hipFree(d_freq);
  if (hf) hipHostFree(hf);
  if (n_updates) *n_updates = updates;
  return rc;
}

int coding_args(trace_model* m, int32_t B, int64_t length, int64_t stride, int32_t mode) {
  if (!m) return fail(TRACE_EINVAL, "model is NULL");
  if (B < 1 || length < 0 || stride < length) return fail(TRACE_EINVAL, "bad stream count, length or stride");
  if (mode < 0 || mode > 2) return fail(TRACE_EINVAL, "mode must be 0 (never), 1 (gated) or 2 (always)");
  if (B > m->max_windows || (mode != 0 && B > m->max_keep))
    return fail(TRACE_EINVAL, "n_streams above max_windows (or above max_keep when updates are on)");
  return TRACE_OK;
}

// coded length of byte x under one frequency row, log2(total) - log2(freq[x])
double coded_bits(const uint16_t* f, int x, uint32_t* cum_out, uint32_t* tot_out) {
  uint32_t cum = 0, tot = 0;
  for (int v = 0; v < 256; ++v) {
    if (v < x) cum += f[v];
    tot += f[v];
  }
  *cum_out = cum;
  *tot_out = tot;
  return std::log2((double)tot) - std::log2((double)f[x]);
}
}  // namespace

extern "C" int trace_gated_run(trace_model* m, const uint8_t* d_streams, int64_t stride, int32_t n_streams,
                               int64_t pos0, int32_t n_steps, int32_t mode, int32_t ctl_t, double ctl_delta,
                               int32_t max_spec, double* step_ce, int32_t* decisions, int64_t* n_updates,
                               void* stream) {
  if (!m) return fail(TRACE_EINVAL, "model is NULL");
  if (mode < 0 || mode > 2) return fail(TRACE_EINVAL, "mode must be 0 (never), 1 (gated) or 2 (always)");
  if (max_spec < 1) return fail(TRACE_EINVAL, "max_spec must be at least 1");
  if (n_streams < 1) return fail(TRACE_EINVAL, "n_streams must be at least 1");
  int rc = check_windows(m, d_streams, stride, n_streams, pos0, n_steps);
  if (rc) return rc;
  if (mode != 0 && n_streams > m->max_keep) return fail(TRACE_EINVAL, "n_streams above max_keep with updates on");
  trace_controller ctl;
  if (mode == 1 && (rc = trace_controller_init(&ctl, ctl_t, ctl_delta))) return rc;
  if (n_updates) *n_updates = 0;
  if (n_steps == 0) return TRACE_OK;
  const hipStream_t s = S(stream);
  const int32_t spec_max = std::min(max_spec, n_steps);
  float* d_bits = nullptr;
  double *d_ce = nullptr, *h_ce = nullptr;
  hipError_t e = hipMalloc(&d_bits, (size_t)n_streams * spec_max * 4);
  if (e == hipSuccess) e = hipMalloc(&d_ce, (size_t)n_steps * 8);
  if (e == hipSuccess) e = hipHostMalloc((void**)&h_ce, (size_t)n_steps * 8, hipHostMallocDefault);
  rc = e == hipSuccess ? TRACE_OK : fail(TRACE_ENOMEM, "trace_gated_run: buffers");
  const uint32_t tok = TRACE_TOKEN_ATTN;
  int64_t updates = 0;
  int32_t i = 0, spec = 1;
  while (rc == TRACE_OK && i < n_steps) {
    if (mode == 2) {  // always: every step keeps its activations and is updated
      rc = trace_forward_bits(m, d_streams, stride, n_streams, pos0 + i, 1, d_bits, nullptr, d_ce + i,
                              TRACE_KEEP_ACTS | tok, stream);
      if (!rc) rc = trace_adapt_step(m, stream);
      if (decisions) decisions[i] = 1;
      ++updates;
      ++i;
      continue;
    }
    const int32_t S_ = mode == 0 ? std::min(spec_max, n_steps - i) : std::min(spec, n_steps - i);
    rc = trace_forward_bits(m, d_streams, stride, n_streams, pos0 + i, S_, d_bits, nullptr, d_ce + i, tok, stream);
    if (rc) break;
    if (mode == 0) {
      for (int32_t q = 0; q < S_ && decisions; ++q) decisions[i + q] = 0;
      i += S_;
      continue;
    }
    // the controller walks the speculated steps; the weights do not change
    // before the first step it flags, so these are the values it would see
    // one step at a time
    e = hipMemcpyAsync(h_ce + i, d_ce + i, (size_t)S_ * 8, hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) {
      rc = hip_fail(e, "trace_gated_run: step cross-entropies");
      break;
    }
    int32_t used = S_, upd = 0;
    for (int32_t q = 0; q < S_; ++q) {
      rc = trace_controller_decide(&ctl, h_ce[i + q], &upd);
      if (rc) break;
      if (decisions) decisions[i + q] = upd;
      if (upd) {
        used = q + 1;
        break;
      }
    }
    if (rc) break;
    if (upd) {  // Alg. 1 line 10 on the flagged step's batch
      rc = trace_forward_bits(m, d_streams, stride, n_streams, pos0 + i + used - 1, 1, d_bits, nullptr, nullptr,
                              TRACE_KEEP_ACTS | tok, stream);
      if (!rc) rc = trace_adapt_step(m, stream);
      ++updates;
      spec = 1;
    } else {
      spec = std::min(spec_max, 2 * spec);
    }
    i += used;
  }
  if (rc == TRACE_OK && step_ce) {
    e = hipMemcpyAsync(h_ce, d_ce, (size_t)n_steps * 8, hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e == hipSuccess)
      std::memcpy(step_ce, h_ce, (size_t)n_steps * 8);
    else
      rc = hip_fail(e, "trace_gated_run: step cross-entropies");
  }
  if (rc == TRACE_OK) {
    e = hipStreamSynchronize(s);
    if (e != hipSuccess) rc = hip_fail(e, "trace_gated_run");
  } else {
    (void)hipStreamSynchronize(s);
  }
  (void)hipFree(d_bits);
  (void)hipFree(d_ce);
  if (h_ce) (void)hipHostFree(h_ce);
  if (n_updates) *n_updates = updates;
  return rc;
}

extern "C" int trace_compress(trace_model* m, const uint8_t* d_streams, int64_t stride, int32_t n_streams,
                              int64_t length, int32_t mode, int32_t ctl_t, double ctl_delta, uint8_t* out,
                              int64_t out_stride, int64_t* out_sizes, int64_t* n_updates, void* stream) {
  int rc = coding_args(m, n_streams, length, stride, mode);
  if (rc) return rc;
  if (!d_streams || !out || !out_sizes || out_stride < 1) return fail(TRACE_EINVAL, "NULL buffer or out_stride < 1");
  const int32_t B = n_streams;
  std::vector<uint8_t> h((size_t)B * length);
  hipStream_t s = (hipStream_t)stream;
  if (length > 0) {
    // rows packed on the device, then one copy (a strided copy to the host
    // moves row by row)
    uint8_t* d_pack = nullptr;
    hipError_t e = stride == length ? hipSuccess : hipMalloc(&d_pack, (size_t)B * length);
    if (e == hipSuccess && d_pack)
      e = hipMemcpy2DAsync(d_pack, length, d_streams, stride, length, B, hipMemcpyDeviceToDevice, s);
    if (e == hipSuccess)
      e = hipMemcpyAsync(h.data(), d_pack ? d_pack : d_streams, (size_t)B * length, hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (d_pack) hipFree(d_pack);
    if (e != hipSuccess) return hip_fail(e, "trace_compress");
  }
  std::vector<RcEnc> enc(B);
  for (int32_t b = 0; b < B; ++b) {
    enc[b].out = out + (int64_t)b * out_stride;
    enc[b].cap = out_stride;
  }
  auto first = [&](int64_t n0) {
    for (int64_t i = 0; i < n0; ++i)
      for (int32_t b = 0; b < B; ++b) enc[b].encode(h[(size_t)b * length + i], 1, 256);
    return TRACE_OK;
  };
  std::vector<double> cb(B);
  WorkPool pool(B);
  auto code = [&](int64_t i, const uint16_t* hf, double* ce) {
    pool.run(B, [&](int64_t b0, int64_t b1) {
      for (int64_t b = b0; b < b1; ++b) {
        const int x = h[(size_t)b * length + i];
        uint32_t cum, tot;
        cb[b] = coded_bits(hf + (size_t)b * 256, x, &cum, &tot);
        enc[b].encode(cum, hf[(size_t)b * 256 + x], tot);
      }
    });
    for (int32_t b = 0; b < B; ++b) *ce += cb[b];  // streams in order
    return TRACE_OK;
  };
  rc = coding_loop(m, d_streams, stride, B, length, mode, ctl_t, ctl_delta, n_updates, stream, first, code);
  if (rc) return rc;
  bool over = false;
  for (int32_t b = 0; b < B; ++b) {
    enc[b].finish();
    out_sizes[b] = enc[b].n;
    over = over || enc[b].over();
  }
  return over ? fail(TRACE_EINVAL, "out_stride is too small for a code (out_sizes hold the lengths needed)")
              : TRACE_OK;
}

extern "C" int trace_decompress(trace_model* m, const uint8_t* comp, int64_t comp_stride, const int64_t* comp_sizes,
                                int32_t n_streams, int64_t length, int32_t mode, int32_t ctl_t, double ctl_delta,
                                uint8_t* d_out, int64_t stride, int64_t* n_updates, void* stream) {
  int rc = coding_args(m, n_streams, length, stride, mode);
  if (rc) return rc;
  if (!comp || !comp_sizes || !d_out) return fail(TRACE_EINVAL, "NULL buffer");
  const int32_t B = n_streams;
  for (int32_t b = 0; b < B; ++b)
    if (comp_sizes[b] < 0 || comp_sizes[b] > comp_stride) return fail(TRACE_EINVAL, "comp_sizes out of range");
  std::vector<uint8_t> h((size_t)B * std::max<int64_t>(length, 1));
  std::vector<RcDec> dec(B);
  for (int32_t b = 0; b < B; ++b) {
    dec[b].in = comp + (int64_t)b * comp_stride;
    dec[b].size = comp_sizes[b];
    dec[b].start();
  }
  hipStream_t s = (hipStream_t)stream;
  // columns [i0, i0 + n) of the host copy -> d_out: each column as one
  // contiguous copy and a scatter into the rows (strided copies of single
  // bytes are slow)
  // (pinned, so the copy reads it directly; it is rewritten only after the
  // next position's synchronisation, which follows this copy on the stream)
  uint8_t* d_col = nullptr;
  uint8_t* col = nullptr;
  hipError_t e0 = hipMalloc(&d_col, (size_t)B);
  if (e0 == hipSuccess) e0 = hipHostMalloc((void**)&col, (size_t)B, hipHostMallocDefault);
  if (e0 != hipSuccess) {
    if (d_col) hipFree(d_col);
    return hip_fail(e0, "trace_decompress");
  }
  auto put_cols = [&](int64_t i0, int64_t n, bool wait) {
    hipError_t e = hipSuccess;
    for (int64_t i = i0; i < i0 + n && e == hipSuccess; ++i) {
      for (int32_t b = 0; b < B; ++b) col[b] = h[(size_t)b * length + i];
      e = hipMemcpyAsync(d_col, col, (size_t)B, hipMemcpyHostToDevice, s);
      if (e == hipSuccess) {
        launch_put_column(d_col, B, d_out, stride, i, s);
        e = hipGetLastError();
      }
      if (e == hipSuccess && (wait || i + 1 < i0 + n)) e = hipStreamSynchronize(s);
    }
    return e == hipSuccess ? TRACE_OK : hip_fail(e, "trace_decompress");
  };
  auto first = [&](int64_t n0) {
    for (int64_t i = 0; i < n0; ++i)
      for (int32_t b = 0; b < B; ++b) h[(size_t)b * length + i] = (uint8_t)dec[b].decode_uniform();
    return n0 > 0 ? put_cols(0, n0, true) : TRACE_OK;
  };
  std::vector<double> cb(B);
  WorkPool pool(B);
  auto code = [&](int64_t i, const uint16_t* hf, double* ce) {
    pool.run(B, [&](int64_t b0, int64_t b1) {
      for (int64_t b = b0; b < b1; ++b) {
        const uint16_t* f = hf + (size_t)b * 256;
        uint32_t tot = 0;
        for (int v = 0; v < 256; ++v) tot += f[v];
        const int x = dec[b].decode(f, 256, tot);
        h[(size_t)b * length + i] = (uint8_t)x;
        uint32_t cum;
        cb[b] = coded_bits(f, x, &cum, &tot);
      }
    });
    for (int32_t b = 0; b < B; ++b) *ce += cb[b];  // streams in order
    return put_cols(i, 1, false);
  };
  rc = coding_loop(m, d_out, stride, B, length, mode, ctl_t, ctl_delta, n_updates, stream, first, code);
  const hipError_t e1 = hipStreamSynchronize(s);  // the last column's copy reads col
  hipFree(d_col);
  hipHostFree(col);
  if (rc == TRACE_OK && e1 != hipSuccess) rc = hip_fail(e1, "trace_decompress");
  return rc;
}
