// Offline weight preparation (Sec. 4.2): fold the channel scaling into the
// weight (W' = D W), quantize each group of w_group input channels of every
// output channel to symmetric int4 (Eq. 1 with q_max = 7) with an fp16 step,
// and pack two codes per byte.
//
// One wave per (output channel, group): lanes stride over 8-element chunks, so
// every global read is a coalesced 32-byte segment per lane.
#include "sq_internal.h"

namespace sq {
namespace {

__global__ __launch_bounds__(256) void pack_weights_kernel(PackArgs a) {
  const int lane = threadIdx.x & 63;
  const int ng = a.K / a.w_group;
  const long wave = static_cast<long>(flat_wg()) * 4 + (threadIdx.x >> 6);
  if (wave >= static_cast<long>(a.N) * ng) return;
  const int j = static_cast<int>(wave / ng);
  const int b = static_cast<int>(wave % ng);
  const int k0 = b * a.w_group;
  const float* wr = a.w + static_cast<size_t>(j) * a.K + k0;
  const int nchunk = a.w_group / 8;

  float m = 0.0f;
  for (int c = lane; c < nchunk; c += 64) {
    const float4 w0 = *reinterpret_cast<const float4*>(wr + c * 8);
    const float4 w1 = *reinterpret_cast<const float4*>(wr + c * 8 + 4);
    float e[8] = {w0.x, w0.y, w0.z, w0.w, w1.x, w1.y, w1.z, w1.w};
    if (a.d != nullptr) {
      const float4 d0 = *reinterpret_cast<const float4*>(a.d + k0 + c * 8);
      const float4 d1 = *reinterpret_cast<const float4*>(a.d + k0 + c * 8 + 4);
      const float dd[8] = {d0.x, d0.y, d0.z, d0.w, d1.x, d1.y, d1.z, d1.w};
#pragma unroll
      for (int i = 0; i < 8; ++i) e[i] *= dd[i];
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) m = fmaxf(m, fabsf(e[i]));
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) m = fmaxf(m, __shfl_xor(m, o, 64));

  const uint32_t sbits = f32_to_f16(m / 7.0f);
  float inv = 1.0f / f16_to_f32(sbits);
  if (__builtin_isinf(inv)) inv = 0.0f;

  uint8_t* qr = a.qw + static_cast<size_t>(j) * (a.K / 2) + k0 / 2;
  for (int c = lane; c < nchunk; c += 64) {
    const float4 w0 = *reinterpret_cast<const float4*>(wr + c * 8);
    const float4 w1 = *reinterpret_cast<const float4*>(wr + c * 8 + 4);
    float e[8] = {w0.x, w0.y, w0.z, w0.w, w1.x, w1.y, w1.z, w1.w};
    if (a.d != nullptr) {
      const float4 d0 = *reinterpret_cast<const float4*>(a.d + k0 + c * 8);
      const float4 d1 = *reinterpret_cast<const float4*>(a.d + k0 + c * 8 + 4);
      const float dd[8] = {d0.x, d0.y, d0.z, d0.w, d1.x, d1.y, d1.z, d1.w};
#pragma unroll
      for (int i = 0; i < 8; ++i) e[i] *= dd[i];
    }
    uint32_t word = 0u;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      float t = e[i] * inv;
      t = fminf(fmaxf(t, -7.0f), 7.0f);
      const int q = static_cast<int>(__builtin_rintf(t));
      word |= (static_cast<uint32_t>(q) & 0xFu) << (8 * (i & 3) + 4 * (i >> 2));
    }
    *reinterpret_cast<uint32_t*>(qr + c * 4) = word;
  }
  if (lane == 0) a.w_scale[static_cast<size_t>(b) * a.N + j] = static_cast<uint16_t>(sbits);  // group-major
}

}  // namespace

hipError_t launch_pack_weights(const PackArgs& a, hipStream_t s) {
  const long waves = static_cast<long>(a.N) * (a.K / a.w_group);
  hipLaunchKernelGGL(pack_weights_kernel, wg_grid(static_cast<size_t>((waves + 3) / 4)), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace sq
