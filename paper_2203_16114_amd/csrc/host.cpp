// Host-only parts of libtrace: configuration checks, the canonical parameter
// layout, the seeded initialiser (Model.initialize of Alg. 1) and the
// back-prop controller (Sec. 4.4, Algorithm 2, Eq. 7).  No GPU is touched here.
// Built without floating-point contraction so the double-precision
// Box-Muller draws and the controller threshold are plain IEEE operations.
#include <cmath>
#include <cstdint>
#include <cstring>
#include <string>

#include "../../include/trace.h"
#include "host.h"

static thread_local std::string g_last_error;

void trace_set_error(const std::string& msg) { g_last_error = msg; }
extern "C" const char* trace_last_error(void) { return g_last_error.c_str(); }

extern "C" const char* trace_strerror(int code) {
  switch (code) {
    case TRACE_OK: return "ok";
    case TRACE_EINVAL: return "invalid argument";
    case TRACE_ENOMEM: return "out of memory";
    case TRACE_EHIP: return "HIP runtime error";
    case TRACE_ESTATE: return "call out of order";
    case TRACE_ENONFINITE: return "non-finite cross-entropy";
    case TRACE_EUNSUPPORTED: return "no kernel built for this shape";
    default: return "unknown error";
  }
}

int trace_check_config(const trace_config* c, Layout* L) {
  if (!c) {
    trace_set_error("config is NULL");
    return TRACE_EINVAL;
  }
  if (c->W <= 0 || c->e <= 0 || c->g <= 0 || c->H <= 0 || c->F <= 0 || c->k <= 0) {
    trace_set_error("W, e, g, H, F and k must be positive");
    return TRACE_EINVAL;
  }
  if (c->W % c->g != 0) {
    trace_set_error("W must be a multiple of g");
    return TRACE_EINVAL;
  }
  const int64_t d = (int64_t)c->g * c->e;
  if (d % c->H != 0) {
    trace_set_error("d = g*e must be a multiple of H");
    return TRACE_EINVAL;
  }
  if (c->dtype != TRACE_FP32 && c->dtype != TRACE_BF16) {
    trace_set_error("dtype must be TRACE_FP32 or TRACE_BF16");
    return TRACE_EINVAL;
  }
  if (c->use_pos != 0 && c->use_pos != 1) {
    trace_set_error("use_pos must be 0 or 1");
    return TRACE_EINVAL;
  }
  if (c->k > 8) {
    trace_set_error("k must be at most 8");
    return TRACE_EINVAL;
  }
  if (c->max_windows < 0 || c->max_keep < 0) {
    trace_set_error("max_windows and max_keep must be non-negative");
    return TRACE_EINVAL;
  }
  if (c->untied_ffn != 0 && c->untied_ffn != 1) {
    trace_set_error("untied_ffn must be 0 or 1");
    return TRACE_EINVAL;
  }
  if (c->attention != TRACE_ATTN_SOFTMAX && c->attention != TRACE_ATTN_PERFORMER) {
    trace_set_error("attention must be TRACE_ATTN_SOFTMAX or TRACE_ATTN_PERFORMER");
    return TRACE_EINVAL;
  }
  if (c->layers < 0 || c->layers > 8) {
    trace_set_error("layers must be in [0, 8] (0: one layer)");
    return TRACE_EINVAL;
  }
  if (c->layers > 1 && c->attention != TRACE_ATTN_SOFTMAX) {
    trace_set_error("stacked layers use softmax attention");
    return TRACE_EINVAL;
  }
  if (c->n_features < 0 || c->n_features > 512 || c->n_features % 16 != 0) {
    trace_set_error("n_features must be a multiple of 16 in [0, 512]");
    return TRACE_EINVAL;
  }
  if (!(c->lr >= 0.0) || !(c->beta1 >= 0.0 && c->beta1 < 1.0) || !(c->beta2 >= 0.0 && c->beta2 < 1.0) ||
      !(c->eps > 0.0)) {
    trace_set_error("Adam settings out of range (lr >= 0, 0 <= beta < 1, eps > 0)");
    return TRACE_EINVAL;
  }
  if (L) {
    L->T = c->W / c->g;
    L->D = (int)d;
    L->DH = (int)(d / c->H);
    const int64_t T = L->T, D = d, e = c->e, F = c->F;
    const int64_t nr = c->untied_ffn ? c->k : 1;  // FFN weight blocks: one, or one per repeat
    const int64_t NL = c->layers > 1 ? c->layers : 1;
    L->NL = (int)NL;
    const int64_t sizes[NPARAM] = {256 * e, T * D, D * D, D * D, D * D, D * D, nr * D * F, nr * F * D, D * 256, 256};
    int64_t off = 0;
    for (int i = 0; i < NPARAM; ++i) {
      const bool per_layer = i >= P_WQ && i <= P_W2;
      L->off[i] = off;
      L->lsize[i] = sizes[i];
      L->size[i] = per_layer ? NL * sizes[i] : sizes[i];
      off += L->size[i];
    }
    L->n = off;
  }
  return TRACE_OK;
}

extern "C" int trace_param_count(const trace_config* cfg, int64_t* n) {
  if (!n) {
    trace_set_error("n is NULL");
    return TRACE_EINVAL;
  }
  Layout L;
  const int rc = trace_check_config(cfg, &L);
  if (rc) return rc;
  *n = L.n;
  return TRACE_OK;
}

// splitmix64 (Vigna): one step of the state and its output.
static inline uint64_t splitmix64_next(uint64_t* s) {
  uint64_t z = (*s += 0x9E3779B97F4A7C15ULL);
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

void trace_fill_init(const Layout& L, uint64_t seed, double stdv, float* out) {
  const int64_t n_rand = L.n - 256;  // bout (last) starts at zero
  uint64_t state = seed;
  const double two_pi = 2.0 * 3.141592653589793;
  for (int64_t i = 0; i < n_rand; i += 2) {
    const uint64_t x1 = splitmix64_next(&state);
    const uint64_t x2 = splitmix64_next(&state);
    const double u1 = ((double)(x1 >> 11) + 0.5) * 0x1.0p-53;
    const double u2 = ((double)(x2 >> 11) + 0.5) * 0x1.0p-53;
    const double r = std::sqrt(-2.0 * std::log(u1));
    out[i] = (float)(stdv * (r * std::cos(two_pi * u2)));
    if (i + 1 < n_rand) out[i + 1] = (float)(stdv * (r * std::sin(two_pi * u2)));
  }
  for (int64_t i = n_rand; i < L.n; ++i) out[i] = 0.f;
}

extern "C" int trace_init_flat_host(const trace_config* cfg, uint64_t seed, double stdv, float* host_out, int64_t n) {
  Layout L;
  const int rc = trace_check_config(cfg, &L);
  if (rc) return rc;
  if (!host_out || n != L.n) {
    trace_set_error("host_out must hold trace_param_count floats");
    return TRACE_EINVAL;
  }
  if (!std::isfinite(stdv)) {
    trace_set_error("std must be finite");
    return TRACE_EINVAL;
  }
  trace_fill_init(L, seed, stdv, host_out);
  return TRACE_OK;
}

// ------------------------------------------------------------- controller ----
extern "C" int trace_controller_init(trace_controller* c, int32_t t, double delta) {
  if (!c) {
    trace_set_error("controller is NULL");
    return TRACE_EINVAL;
  }
  if (t < 1 || t > 256) {
    trace_set_error("cache size t must be in 1..256");
    return TRACE_EINVAL;
  }
  if (!std::isfinite(delta)) {
    trace_set_error("delta must be finite");
    return TRACE_EINVAL;
  }
  std::memset(c, 0, sizeof(*c));
  c->t = t;
  c->delta = delta;
  c->sum = 0.0;
  return TRACE_OK;
}

extern "C" int trace_controller_decide(trace_controller* c, double e, int32_t* update) {
  if (!c || !update) {
    trace_set_error("controller or update is NULL");
    return TRACE_EINVAL;
  }
  *update = 0;
  if (c->t < 1 || c->t > 256 || c->count < 0 || c->count > c->t || c->head < 0 || c->head >= c->t) {
    trace_set_error("controller not initialised");
    return TRACE_EINVAL;
  }
  if (!std::isfinite(e)) {
    trace_set_error("non-finite cross-entropy");
    return TRACE_ENONFINITE;
  }
  // Alg. 2 lines 4-8 with the prose reading of Sec. 4.4: back-propagate when the
  // current entropy exceeds the cache mean (Eq. 7) by more than delta; while the
  // cache is still filling, always back-propagate.
  int32_t upd;
  if (c->count < c->t)
    upd = 1;
  else
    upd = (e > (c->sum / (double)c->t + c->delta)) ? 1 : 0;
  // Alg. 2 lines 10-11: the oldest entry leaves a full cache, e enters it.
  if (c->count == c->t) {
    c->sum = c->sum - c->ring[c->head];
    c->ring[c->head] = e;
    c->head = (c->head + 1) % c->t;
  } else {
    c->ring[(c->head + c->count) % c->t] = e;
    c->count += 1;
  }
  c->sum = c->sum + e;
  *update = upd;
  return TRACE_OK;
}
