// Measurement hook: the int8 matrix-core rate this GPU sustains, as a ceiling
// to set beside the published peak.  Every wave of a full-occupancy grid (two
// 256-thread workgroups per CU, as the tiled GEMM runs) issues back-to-back
// v_mfma_i32_32x32x32_i8 on register operands, with no memory traffic in the
// loop.  Operands all zero or pseudo-random: the rate depends on the data
// (random operands draw more power).  With `fold`, each 32x32 tile's
// accumulator is also converted and multiply-added into fp32 once per four
// MFMAs, the dequantization work per 128-channel block of the GEMM.
#include "sq_internal.h"

namespace sq {
namespace {

typedef int v4i_p __attribute__((ext_vector_type(4)));
typedef int v16i_p __attribute__((ext_vector_type(16)));

template <bool FOLD>
__global__ __launch_bounds__(256, 2) void mfma_probe_kernel(int32_t* sink, int32_t iters, int32_t random) {
  const int l = threadIdx.x & 63;
  v4i_p a[4], b[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    uint32_t h = (static_cast<uint32_t>(l) * 4 + i) * 2654435761u + blockIdx.x * 97u;
    h ^= h >> 13;
    h *= 2246822519u;
    h ^= h >> 16;
    const int m = random ? -1 : 0;
    a[i] = (v4i_p){static_cast<int>(h) & m, static_cast<int>(h * 3u) & m, static_cast<int>(h * 5u) & m,
                   static_cast<int>(h * 7u) & m};
    b[i] = (v4i_p){static_cast<int>(h * 11u) & m, static_cast<int>(h * 13u) & m, static_cast<int>(h * 17u) & m,
                   static_cast<int>(h * 19u) & m};
  }
  v16i_p acc[4];
  float y[4][16];
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    acc[t] = (v16i_p)(0);
#pragma unroll
    for (int r = 0; r < 16; ++r) y[t][r] = 0.0f;
  }
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      if constexpr (FOLD) {
#pragma unroll
        for (int r = 0; r < 16; ++r) y[t][r] = __builtin_fmaf(static_cast<float>(acc[t][r]), 0.001f, y[t][r]);
        acc[t] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a[0], b[t], (v16i_p)(0), 0, 0, 0);
      } else {
        acc[t] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a[0], b[t], acc[t], 0, 0, 0);
      }
#pragma unroll
      for (int s = 1; s < 4; ++s)
        acc[t] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a[s], b[(t + s) & 3], acc[t], 0, 0, 0);
    }
  }
  int s = 0;
#pragma unroll
  for (int t = 0; t < 4; ++t)
#pragma unroll
    for (int r = 0; r < 16; ++r) s += acc[t][r] + static_cast<int>(y[t][r]);
  sink[blockIdx.x * 256 + threadIdx.x] = s;  // keeps the work live
}

}  // namespace

int mfma_probe_workgroups() { return device_cus() * 2; }

hipError_t launch_mfma_probe(int32_t* sink, int32_t iters, int32_t random, int32_t fold, hipStream_t s) {
  const dim3 grid(static_cast<unsigned>(mfma_probe_workgroups()));
  if (fold)
    hipLaunchKernelGGL((mfma_probe_kernel<true>), grid, dim3(256), 0, s, sink, iters, random);
  else
    hipLaunchKernelGGL((mfma_probe_kernel<false>), grid, dim3(256), 0, s, sink, iters, random);
  return hipGetLastError();
}

}  // namespace sq
