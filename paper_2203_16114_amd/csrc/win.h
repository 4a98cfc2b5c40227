// Byte offset of the target of window n_local of a launch (device code).
#pragma once
#include "kernels.h"

__device__ __forceinline__ int64_t target_offset(const WinArgs& w, int64_t n_local) {
  const int64_t gn = w.n0 + n_local;
  const int64_t b = gn / w.n_steps;
  const int64_t s = gn - b * w.n_steps;
  return b * w.stride + w.pos0 + s;
}
