// trace_forward_bits_noalloc: the forward estimator for callers that cannot
// allocate device memory.  Its one workspace, the fp32 hand-off h0 = Attn + X
// between the attention and FFN kernels, is the fixed array `scratch` below
// instead of the model's allocated buffer; the launches are those of
// trace_forward_bits.
#include <hip/hip_runtime.h>

#include <mutex>
#include <string>

#include "../../include/trace.h"
#include "host.h"

namespace {

constexpr int64_t kScratchBytes = (int64_t)32 << 20;
constexpr int kMaxDevices = 64;

std::mutex g_mu;
void* g_scratch[kMaxDevices];  // address of `scratch` on each device, once resolved

}  // namespace

// One copy per device, held until the process ends.  In host code the name is
// a host-side stand-in: only the address from hipGetSymbolAddress is passed on.
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

int trace_scratch_setup(int device) {
  if (device < 0 || device >= kMaxDevices) {
    trace_set_error("device ordinal out of range for the fixed workspace");
    return TRACE_EINVAL;
  }
  std::lock_guard<std::mutex> lk(g_mu);
  if (g_scratch[device]) return TRACE_OK;
  void* p = nullptr;
  const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
  if (e != hipSuccess || p == nullptr) {
    trace_set_error(std::string("hipGetSymbolAddress(scratch): ") + hipGetErrorString(e));
    return TRACE_EHIP;
  }
  g_scratch[device] = p;
  return TRACE_OK;
}

extern "C" int trace_forward_bits_noalloc(trace_model* m, const uint8_t* d_streams, int64_t stride, int32_t n_streams,
                                          int64_t pos0, int32_t n_steps, float* d_bits, float* d_logits,
                                          double* d_step_ce, uint32_t flags, void* stream) {
  if (!m) {
    trace_set_error("model is NULL");
    return TRACE_EINVAL;
  }
  const int dev = trace_model_device(m);
  int cur = -1;
  if (hipGetDevice(&cur) != hipSuccess || cur != dev) {
    trace_set_error("trace_forward_bits_noalloc: the model's device must be current");
    return TRACE_EINVAL;
  }
  const int64_t cap = kScratchBytes / (4 * (int64_t)trace_model_dim(m));
  if (n_streams > 0 && n_steps > 0 && (int64_t)n_streams * n_steps > cap) {
    trace_set_error("trace_forward_bits_noalloc: " + std::to_string((int64_t)n_streams * n_steps) +
                    " windows exceed the fixed workspace (" + std::to_string(cap) + " windows of this model)");
    return TRACE_EINVAL;
  }
  int rc = trace_scratch_setup(dev);  // resolved by trace_create; retried here if that failed
  if (rc) return rc;
  void* ws;
  {
    std::lock_guard<std::mutex> lk(g_mu);
    ws = g_scratch[dev];
  }
  return trace_forward_into(m, d_streams, stride, n_streams, pos0, n_steps, d_bits, d_logits, d_step_ce, flags, stream,
                            (float*)ws, cap, false);
}
