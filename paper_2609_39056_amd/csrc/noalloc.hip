// The allocation-free variant of the fused W4A8 linear: the workspace that
// sq_linear_w4a8 takes from the caller (Q_X, the row scales and the split-K
// partial sums) lives instead in one file-scope device array of this library,
// so a caller that cannot allocate device memory (code under HIP graph
// capture, tight serving loops, harnesses that forbid hipMalloc) passes only
// its inputs and output.
#include <mutex>

#include "sq_internal.h"

namespace sq {
namespace {

// One copy per GPU, held until the process ends.  Host code never passes
// `scratch` itself to a kernel or a copy: in host code the name is a stand-in
// for the device symbol, and its device address comes from
// hipGetSymbolAddress (per device, below).
static __device__ __align__(256) uint8_t scratch[SQ_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_mutex;
void* g_scratch_ptr[kMaxDevices];  // device address of `scratch` on each device, once looked up

// The device address of this device's scratch array, looked up once per
// device with that device current; nullptr on failure.
void* scratch_ptr() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lock(g_mutex);
  if (g_scratch_ptr[dev] == nullptr) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr) return nullptr;
    g_scratch_ptr[dev] = p;
  }
  return g_scratch_ptr[dev];
}

}  // namespace
}  // namespace sq

extern "C" sq_status sq_linear_w4a8_noalloc(const uint16_t* x, int32_t M, const sq_act_params* act,
                                            const sq_weight* w, void* y, int32_t out_dtype, hipStream_t stream) {
  void* ws = sq::scratch_ptr();
  if (ws == nullptr) return SQ_ERR_HIP;
  // the usual validation, in the usual order; a layer whose workspace exceeds
  // the array returns SQ_ERR_WORKSPACE before anything is launched
  return sq::linear_fused_on(8, x, M, act, w, y, out_dtype, ws, SQ_NOALLOC_SCRATCH_BYTES, stream);
}
