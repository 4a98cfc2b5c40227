// Host-side helpers shared by host.cpp and api.cpp.
#pragma once
#include <cstdint>
#include <string>

#include "../../include/trace.h"

// canonical flat parameter order
enum { P_E = 0, P_P, P_WQ, P_WK, P_WV, P_WO, P_W1, P_W2, P_WOUT, P_BOUT, NPARAM };

struct Layout {
  int T, D, DH;
  int64_t off[NPARAM], size[NPARAM], n;
};

void trace_set_error(const std::string& msg);
int trace_check_config(const trace_config* c, Layout* L);
void trace_fill_init(const Layout& L, uint64_t seed, double stdv, float* out);
