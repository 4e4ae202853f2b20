// Measurement hook: the int8 matrix-core rate this GPU sustains, as a ceiling
// to set beside the published peak.  Every wave of a full-occupancy grid (two
// 256-thread workgroups per CU, as the tiled GEMM runs) issues back-to-back
// int8 MFMAs on register operands, with no memory traffic in the loop, in
// either of the two forms the GEMM kernels use:
//  - v_mfma_i32_32x32x32_i8, four 32 x 32 tiles of four MFMAs per iteration;
//    with `fold`, each tile's accumulator is converted (v_cvt_f32_i32) and
//    multiply-added into fp32 once per four MFMAs, the dequantization of one
//    128-channel block;
//  - v_mfma_i32_16x16x64_i8, sixteen 16 x 16 tiles of two MFMAs per
//    iteration (a wave's 64 x 64 outputs over one 128-channel stage); with
//    `fold`, each block starts from the integer bits of 1.5 * 2^23 and is
//    folded by a subtraction and an fma per output, the tiled 16 x 16 kernel's
//    biased fold.
// Both issue 2^20 int8 operations per wave and iteration.  Operands all zero
// or pseudo-random: the rate depends on the data (random operands draw more
// power).  A third probe runs the 4-bit path's fp8 / fp6 instruction.
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

template <bool FOLD>
__global__ __launch_bounds__(256, 2) void mfma_probe16_kernel(int32_t* sink, int32_t iters, int32_t random) {
  const int l = threadIdx.x & 63;
  v4i_p a[2], b[4][2];
  {
    uint32_t h = static_cast<uint32_t>(l) * 2654435761u + blockIdx.x * 97u;
    const int m = random ? -1 : 0;
    auto next = [&]() {
      h ^= h >> 13;
      h *= 2246822519u;
      h ^= h >> 16;
      h += 0x9E3779B9u;
      return static_cast<int>(h) & m;
    };
#pragma unroll
    for (int i = 0; i < 2; ++i) a[i] = (v4i_p){next(), next(), next(), next()};
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int i = 0; i < 2; ++i) b[t][i] = (v4i_p){next(), next(), next(), next()};
  }
  constexpr int kMagic = 0x4B400000;  // the bits of 1.5 * 2^23
  const v4i_p magic = (v4i_p)(FOLD ? kMagic : 0);
  v4i_p acc[16];
  float y[16][4];
#pragma unroll
  for (int t = 0; t < 16; ++t) {
    acc[t] = magic;
#pragma unroll
    for (int r = 0; r < 4; ++r) y[t][r] = 0.0f;
  }
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int t = 0; t < 16; ++t) {
      if constexpr (FOLD) {
#pragma unroll
        for (int r = 0; r < 4; ++r) y[t][r] = __builtin_fmaf(__int_as_float(acc[t][r]) - 12582912.0f, 0.001f, y[t][r]);
        acc[t] = __builtin_amdgcn_mfma_i32_16x16x64_i8(a[0], b[t & 3][0], magic, 0, 0, 0);
      } else {
        acc[t] = __builtin_amdgcn_mfma_i32_16x16x64_i8(a[0], b[t & 3][0], acc[t], 0, 0, 0);
      }
      acc[t] = __builtin_amdgcn_mfma_i32_16x16x64_i8(a[1], b[(t >> 2) & 3][1], acc[t], 0, 0, 0);
    }
  }
  int s = 0;
#pragma unroll
  for (int t = 0; t < 16; ++t)
#pragma unroll
    for (int r = 0; r < 4; ++r) s += acc[t][r] + static_cast<int>(y[t][r]);
  sink[blockIdx.x * 256 + threadIdx.x] = s;  // keeps the work live
}

// The 4-bit path's instruction, v_mfma_scale_f32_32x32x64_f8f6f4, on fp8
// (e4m3) or fp6 (e2m3) operands: per iteration a wave issues the eight MFMAs
// of one 128-channel stage of the fp8 W4A4 kernel (2 x 2 tiles of 32 x 32,
// two 64-wide blocks), 2^20 operations.  With `fold`, each block's fp32 sum is
// folded as that kernel does: two fmas per output (the group step with its
// offset term, then the weight step).  fp6 operands take six of the eight
// operand registers (32 six-bit codes per lane).
template <int FMT, bool FOLD>
__global__ __launch_bounds__(256, 2) void mfma_probe_f8f6_kernel(int32_t* sink, int32_t iters, int32_t random) {
  typedef int v8i_p __attribute__((ext_vector_type(8)));
  typedef float v16f_p __attribute__((ext_vector_type(16)));
  const int l = threadIdx.x & 63;
  v8i_p a[2], b[2];  // one operand per row tile and per column tile (both blocks reuse them)
  {
    uint32_t h = static_cast<uint32_t>(l) * 2654435761u + blockIdx.x * 97u;
    // random bits; fp8 bytes masked to exponents below 15 (no NaN encodings)
    const uint32_t m = random ? (FMT == 8 ? 0x6F6F6F6Fu : 0xFFFFFFFFu) : 0u;
    auto next = [&]() {
      h ^= h >> 13;
      h *= 2246822519u;
      h ^= h >> 16;
      h += 0x9E3779B9u;
      return static_cast<int>(h & m);
    };
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      a[i] = (v8i_p){next(), next(), next(), next(), next(), next(), next(), next()};
      b[i] = (v8i_p){next(), next(), next(), next(), next(), next(), next(), next()};
    }
  }
  constexpr int kFmt = FMT == 8 ? 0 : 2;  // operand format: fp8 e4m3 or fp6 e2m3
  v16f_p acc[4];
  float y[4][16];
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    acc[t] = (v16f_p)(0.0f);
#pragma unroll
    for (int r = 0; r < 16; ++r) y[t][r] = 0.0f;
  }
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int hb = 0; hb < 2; ++hb)
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        if constexpr (FOLD) {
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const float u = __builtin_fmaf(acc[t][r], 0.75f, -0.25f);
            y[t][r] = __builtin_fmaf(u, 0.001f, y[t][r]);
          }
          acc[t] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a[t >> 1], b[t & 1], (v16f_p)(0.0f), kFmt,
                                                                    kFmt, 0, 0, 0, 0);
        } else {
          acc[t] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a[t >> 1], b[t & 1], acc[t], kFmt, kFmt,
                                                                    0, 0, 0, 0);
        }
      }
  }
  float s = 0.0f;
#pragma unroll
  for (int t = 0; t < 4; ++t)
#pragma unroll
    for (int r = 0; r < 16; ++r) s += acc[t][r] + y[t][r];
  sink[blockIdx.x * 256 + threadIdx.x] = __float_as_int(s);  // keeps the work live
}

}  // namespace

int mfma_probe_workgroups() { return device_cus() * 2; }

hipError_t launch_mfma_probe_f8f6(int32_t* sink, int32_t fmt, int32_t iters, int32_t random, int32_t fold,
                                  hipStream_t s) {
  const dim3 grid(static_cast<unsigned>(mfma_probe_workgroups()));
  if (fmt == 8) {
    if (fold)
      hipLaunchKernelGGL((mfma_probe_f8f6_kernel<8, true>), grid, dim3(256), 0, s, sink, iters, random);
    else
      hipLaunchKernelGGL((mfma_probe_f8f6_kernel<8, false>), grid, dim3(256), 0, s, sink, iters, random);
  } else if (fold) {
    hipLaunchKernelGGL((mfma_probe_f8f6_kernel<6, true>), grid, dim3(256), 0, s, sink, iters, random);
  } else {
    hipLaunchKernelGGL((mfma_probe_f8f6_kernel<6, false>), grid, dim3(256), 0, s, sink, iters, random);
  }
  return hipGetLastError();
}

hipError_t launch_mfma_probe(int32_t* sink, int32_t shape, int32_t iters, int32_t random, int32_t fold,
                             hipStream_t s) {
  const dim3 grid(static_cast<unsigned>(mfma_probe_workgroups()));
  if (shape == 16) {
    if (fold)
      hipLaunchKernelGGL((mfma_probe16_kernel<true>), grid, dim3(256), 0, s, sink, iters, random);
    else
      hipLaunchKernelGGL((mfma_probe16_kernel<false>), grid, dim3(256), 0, s, sink, iters, random);
  } else if (fold) {
    hipLaunchKernelGGL((mfma_probe_kernel<true>), grid, dim3(256), 0, s, sink, iters, random);
  } else {
    hipLaunchKernelGGL((mfma_probe_kernel<false>), grid, dim3(256), 0, s, sink, iters, random);
  }
  return hipGetLastError();
}

}  // namespace sq
