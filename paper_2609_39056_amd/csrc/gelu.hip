// GELU on bf16 values (the op the quantized DiT keeps in bf16 between the
// MLP's up and down projections, App. D): y = bf16(GELU(x)) with the fp32
// sequence of gelu.h, so that it matches the up projection's GELU epilogue
// bit for bit.  Memory-bound: 16-byte loads and stores, eight values per
// thread, the last partial group element by element.
#include "gelu.h"
#include "sq_internal.h"

namespace sq {
namespace {

constexpr int kPerThread = 8;

__device__ __forceinline__ uint32_t gelu_pair(uint32_t p) {
  float a = gelu_f32(bf16_to_f32(p & 0xFFFFu));
  float b = gelu_f32(bf16_to_f32(p >> 16));
  bf16_round2(a, b);
  return (__float_as_uint(a) >> 16) | (__float_as_uint(b) & 0xFFFF0000u);
}

__global__ __launch_bounds__(256) void gelu_bf16_kernel(const uint16_t* x, size_t n,
                                                       uint16_t* y) {
  const size_t i = (flat_wg() * 256 + threadIdx.x) * kPerThread;
  if (i >= n) return;
  if (i + kPerThread <= n) {
    const uint4 v = *reinterpret_cast<const uint4*>(x + i);
    *reinterpret_cast<uint4*>(y + i) = make_uint4(gelu_pair(v.x), gelu_pair(v.y), gelu_pair(v.z), gelu_pair(v.w));
  } else {
    for (size_t j = i; j < n; ++j) y[j] = static_cast<uint16_t>(gelu_pair(x[j]) & 0xFFFFu);
  }
}

}  // namespace

hipError_t launch_gelu_bf16(const uint16_t* x, size_t n, uint16_t* y, hipStream_t s) {
  if (n == 0) return hipSuccess;
  const size_t groups = (n + 256 * kPerThread - 1) / (256 * kPerThread);
  hipLaunchKernelGGL(gelu_bf16_kernel, wg_grid(groups), dim3(256), 0, s, x, n, y);
  return hipGetLastError();
}

}  // namespace sq
