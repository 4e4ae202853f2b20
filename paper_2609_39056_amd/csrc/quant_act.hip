// The first fused kernel of Sec. 4.4: channel scaling D^-1 (Eq. 6), stream
// gain gamma_{tau,s(i)} (Eq. 8) and symmetric quantization (Eq. 1) in one
// streaming pass over X.  Only the integer codes and the row / group scales are
// written.
//
// Mapping: TPR threads own one row (64 = one wave for K <= 4096, else 256 = the
// whole workgroup); thread t of a row owns 8-element chunks t, t+TPR, ...,
// which stay in registers between the range reduction and the quantization,
// so X is read from HBM exactly once.  A 64-wide 4-bit group is 8 consecutive
// chunks = 8 adjacent lanes, reduced with three lane shuffles.
#include "sq_internal.h"

namespace sq {
namespace {

template <int BITS, int TPR, int NCH>
__global__ __launch_bounds__(256) void quantize_act_kernel(QuantArgs a) {
  constexpr int RPW = 256 / TPR;
  constexpr float QA = BITS == 8 ? 127.0f : 7.0f;
  const int tid = threadIdx.x;
  const int lr = tid % TPR;
  const int row = blockIdx.x * RPW + tid / TPR;
  const bool row_ok = row < a.M;
  const int rowc = row_ok ? row : a.M - 1;
  const int nch = a.K >> 3;
  const bool dynamic = a.range_mode == SQ_RANGE_DYNAMIC;

  const uint16_t* xr = a.x + static_cast<size_t>(rowc) * a.K;
  float v[NCH][8];
#pragma unroll
  for (int j = 0; j < NCH; ++j) {
    const int c = lr + j * TPR;
    if (c < nch) {
      const uint4 raw = *reinterpret_cast<const uint4*>(xr + c * 8);
      const uint32_t wd[4] = {raw.x, raw.y, raw.z, raw.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        v[j][2 * e] = __uint_as_float(wd[e] << 16);
        v[j][2 * e + 1] = __uint_as_float(wd[e] & 0xFFFF0000u);
      }
      if (a.dinv != nullptr) {
        const float4 d0 = *reinterpret_cast<const float4*>(a.dinv + c * 8);
        const float4 d1 = *reinterpret_cast<const float4*>(a.dinv + c * 8 + 4);
        v[j][0] *= d0.x; v[j][1] *= d0.y; v[j][2] *= d0.z; v[j][3] *= d0.w;
        v[j][4] *= d1.x; v[j][5] *= d1.y; v[j][6] *= d1.z; v[j][7] *= d1.w;
      }
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) v[j][e] = 0.0f;
    }
  }

  const float g = a.gamma[a.step * a.S + a.tok2stream[rowc]];
  const float cst = dynamic ? 0.0f : a.clip[a.step];

  // Range c: one per row (8-bit) or one per 64-group (4-bit).
  float cj[BITS == 8 ? 1 : NCH];
  if constexpr (BITS == 8) {
    float m = 0.0f;
    if (dynamic) {
#pragma unroll
      for (int j = 0; j < NCH; ++j)
#pragma unroll
        for (int e = 0; e < 8; ++e) m = fmaxf(m, fabsf(v[j][e]));
#pragma unroll
      for (int o = 32; o >= 1; o >>= 1) m = fmaxf(m, __shfl_xor(m, o, 64));
      if constexpr (TPR > 64) {
        __shared__ float red[TPR / 64];
        if ((tid & 63) == 0) red[tid >> 6] = m;
        __syncthreads();
#pragma unroll
        for (int w = 0; w < TPR / 64; ++w) m = fmaxf(m, red[w]);
      }
    }
    cj[0] = dynamic ? m : cst;
  } else {
#pragma unroll
    for (int j = 0; j < NCH; ++j) {
      float m = 0.0f;
      if (dynamic) {
#pragma unroll
        for (int e = 0; e < 8; ++e) m = fmaxf(m, fabsf(v[j][e]));
        m = fmaxf(m, __shfl_xor(m, 1, 64));
        m = fmaxf(m, __shfl_xor(m, 2, 64));
        m = fmaxf(m, __shfl_xor(m, 4, 64));
      }
      cj[j] = dynamic ? m : cst;
    }
  }
  if (!row_ok) return;

  if constexpr (BITS == 8) {
    const float delta = cj[0] / QA;
    float inv = 1.0f / delta;
    if (__builtin_isinf(inv)) inv = 0.0f;
    int8_t* qr = static_cast<int8_t*>(a.qx) + static_cast<size_t>(row) * a.K;
#pragma unroll
    for (int j = 0; j < NCH; ++j) {
      const int c = lr + j * TPR;
      if (c >= nch) continue;
      uint32_t packed[2] = {0u, 0u};
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        float t = (v[j][e] * g) * inv;
        t = fminf(fmaxf(t, -QA), QA);
        const int q = static_cast<int>(__builtin_rintf(t));
        packed[e >> 2] |= (static_cast<uint32_t>(q) & 0xFFu) << (8 * (e & 3));
      }
      *reinterpret_cast<uint2*>(qr + c * 8) = make_uint2(packed[0], packed[1]);
    }
    if (lr == 0) static_cast<float*>(a.scale)[row] = delta / g;
  } else {
    uint8_t* qr = static_cast<uint8_t*>(a.qx) + static_cast<size_t>(row) * (a.K / 2);
    uint16_t* sr = static_cast<uint16_t*>(a.scale) + static_cast<size_t>(row) * (a.K / kA4Group);
#pragma unroll
    for (int j = 0; j < NCH; ++j) {
      const int c = lr + j * TPR;
      if (c >= nch) continue;
      const uint32_t dbits = f32_to_f16(cj[j] / QA);
      const float delta = f16_to_f32(dbits);
      float inv = 1.0f / delta;
      if (__builtin_isinf(inv)) inv = 0.0f;
      uint32_t word = 0u;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        float t = (v[j][e] * g) * inv;
        t = fminf(fmaxf(t, -QA), QA);
        const int q = static_cast<int>(__builtin_rintf(t));
        // code e < 4 -> low nibble of byte e; code e >= 4 -> high nibble of byte e-4
        word |= (static_cast<uint32_t>(q) & 0xFu) << (8 * (e & 3) + 4 * (e >> 2));
      }
      *reinterpret_cast<uint32_t*>(qr + c * 4) = word;
      if ((c & 7) == 0) sr[c >> 3] = static_cast<uint16_t>(dbits);
    }
  }
}

template <int BITS, int TPR, int NCH>
hipError_t launch_one(const QuantArgs& a, hipStream_t s) {
  constexpr int RPW = 256 / TPR;
  const unsigned grid = static_cast<unsigned>((a.M + RPW - 1) / RPW);
  hipLaunchKernelGGL((quantize_act_kernel<BITS, TPR, NCH>), dim3(grid), dim3(256), 0, s, a);
  return hipGetLastError();
}

template <int BITS>
hipError_t launch_bits(const QuantArgs& a, hipStream_t s) {
  const int nch = a.K / 8;
  if (a.K <= 4096) {
    switch ((nch + 63) / 64) {
      case 1: return launch_one<BITS, 64, 1>(a, s);
      case 2: return launch_one<BITS, 64, 2>(a, s);
      case 3: return launch_one<BITS, 64, 3>(a, s);
      case 4: return launch_one<BITS, 64, 4>(a, s);
      case 5: return launch_one<BITS, 64, 5>(a, s);
      case 6: return launch_one<BITS, 64, 6>(a, s);
      case 7: return launch_one<BITS, 64, 7>(a, s);
      case 8: return launch_one<BITS, 64, 8>(a, s);
      default: return hipErrorInvalidValue;
    }
  }
  switch ((nch + 255) / 256) {
    case 3: return launch_one<BITS, 256, 3>(a, s);
    case 4: return launch_one<BITS, 256, 4>(a, s);
    case 5: return launch_one<BITS, 256, 5>(a, s);
    case 6: return launch_one<BITS, 256, 6>(a, s);
    case 7: return launch_one<BITS, 256, 7>(a, s);
    case 8: return launch_one<BITS, 256, 8>(a, s);
    case 9: return launch_one<BITS, 256, 9>(a, s);
    case 10: return launch_one<BITS, 256, 10>(a, s);
    case 11: return launch_one<BITS, 256, 11>(a, s);
    case 12: return launch_one<BITS, 256, 12>(a, s);
    case 13: return launch_one<BITS, 256, 13>(a, s);
    case 14: return launch_one<BITS, 256, 14>(a, s);
    case 15: return launch_one<BITS, 256, 15>(a, s);
    case 16: return launch_one<BITS, 256, 16>(a, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

hipError_t launch_quantize_act(int act_bits, const QuantArgs& a, hipStream_t s) {
  return act_bits == 8 ? launch_bits<8>(a, s) : launch_bits<4>(a, s);
}

}  // namespace sq
