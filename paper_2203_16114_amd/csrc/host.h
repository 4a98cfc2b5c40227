// Host-side helpers shared by host.cpp and api.cpp.
#pragma once
#include <cstdint>
#include <string>

#include "../../include/trace.h"

// canonical flat parameter order
enum { P_E = 0, P_P, P_WQ, P_WK, P_WV, P_WO, P_W1, P_W2, P_WOUT, P_BOUT, NPARAM };

struct Layout {
  int T, D, DH;
  int NL;                  // layers
  int64_t off[NPARAM], size[NPARAM], n;
  int64_t lsize[NPARAM];   // one layer's block (Wq .. W2); the whole tensor otherwise
  // offset of parameter i of layer l
  int64_t at(int i, int l) const { return off[i] + (int64_t)l * lsize[i]; }
};

void trace_set_error(const std::string& msg);
int trace_check_config(const trace_config* c, Layout* L);
void trace_fill_init(const Layout& L, uint64_t seed, double stdv, float* out);

// Internal entry points shared by api.cpp and noalloc.hip.
struct trace_model;
// The forward of trace_forward_bits with its attention -> FFN hand-off in h0
// (chunks of at most chunk_cap windows); timed = false records no events.
int trace_forward_into(trace_model* m, const uint8_t* d_streams, int64_t stride, int32_t n_streams, int64_t pos0,
                       int32_t n_steps, float* d_bits, float* d_logits, double* d_step_ce, uint32_t flags,
                       void* stream, float* h0, int64_t chunk_cap, bool timed);
int trace_model_dim(const trace_model* m);
int trace_model_device(const trace_model* m);
// Resolves the fixed workspace's address on `device` (which must be current).
int trace_scratch_setup(int device);
