// The first fused kernel of Sec. 4.4: channel scaling D^-1 (Eq. 6), stream
// gain gamma_{tau,s(i)} (Eq. 8) and symmetric quantization (Eq. 1) in one
// streaming pass over X.  Only the integer codes and the row / group scales are
// written.
//
// Mapping: WPR waves (64 * WPR lanes) quantize one row.  Lane l of the row
// owns the 8-element chunks l, l + 64 * WPR, ... (NCH of them), so a 64-wide
// 4-bit group is 8 adjacent lanes.  Every load is issued up front (D^-1, the
// row, then the stream gain); the scaled row stays in registers between the
// range reduction and the quantization, so X is read from HBM exactly once.
// With WPR = 4 the four waves of a workgroup share the row and combine its
// 8-bit range through LDS.
#include "sq_internal.h"

namespace sq {
namespace {

// t rounded to the nearest integer, ties to even, for abs(t) <= 2^22: adding
// 1.5 * 2^23 leaves exactly the rounded value in the low mantissa bits, so the
// two's-complement code is the low byte (8-bit) or nibble (4-bit) of the sum.
__device__ __forceinline__ uint32_t rne_code_bits(float t) { return __float_as_uint(t + 12582912.0f); }

// Bytes b0 of four words, in order, as one word.
__device__ __forceinline__ uint32_t pack_low_bytes(uint32_t w0, uint32_t w1, uint32_t w2, uint32_t w3) {
  const uint32_t lo = __builtin_amdgcn_perm(w1, w0, 0x0c0c0400u);  // [w0.b0, w1.b0, 0, 0]
  const uint32_t hi = __builtin_amdgcn_perm(w3, w2, 0x0c0c0400u);  // [w2.b0, w3.b0, 0, 0]
  return __builtin_amdgcn_perm(hi, lo, 0x05040100u);
}

template <int BITS, int WPR, int NCH, bool F8>
__global__ __launch_bounds__(256) void quantize_act_kernel(QuantArgs a) {
  static_assert(!F8 || BITS == 4, "fp8 code bytes are a 4-bit format");
  static_assert(WPR == 1 || WPR == 4, "a row spans one wave or the whole workgroup");
  constexpr int RPW = 4 / WPR;   // rows per workgroup
  constexpr int LPR = 64 * WPR;  // lanes per row
  constexpr float QA = BITS == 8 ? 127.0f : 7.0f;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lr = (wave % WPR) * 64 + lane;
  const int M = a.M, nch = a.K >> 3;
  const int row = static_cast<int>(flat_wg()) * RPW + wave / WPR;  // past M in the grid's last row: no stores
  const int rowc = min(row, M - 1);
  const bool dynamic = a.range_mode == SQ_RANGE_DYNAMIC;
  const bool has_d = a.dinv != nullptr;

  // D^-1 of the lane's chunks and the row's chunks (clamped inside the matrix)
  float4 d[NCH][2];
  if (has_d) {
#pragma unroll
    for (int j = 0; j < NCH; ++j) {
      const int c = min(lr + j * LPR, nch - 1);
      d[j][0] = *reinterpret_cast<const float4*>(a.dinv + c * 8);
      d[j][1] = *reinterpret_cast<const float4*>(a.dinv + c * 8 + 4);
    }
  }
  const uint16_t* xr = a.x + static_cast<size_t>(rowc) * a.K;
  uint4 raw[NCH];
#pragma unroll
  for (int j = 0; j < NCH; ++j) raw[j] = *reinterpret_cast<const uint4*>(xr + min(lr + j * LPR, nch - 1) * 8);
  const float g = a.gamma[a.step * a.S + a.tok2stream[rowc]];
  const float cst = dynamic ? 0.0f : a.clip[a.step];

  // x~ = X D^-1 (exact bf16 -> fp32 widening, one rounding per product);
  // chunks past the row end hold 0
  float v[NCH][8];
#pragma unroll
  for (int j = 0; j < NCH; ++j) {
    const bool ok = lr + j * LPR < nch;
    const uint32_t wd[4] = {raw[j].x, raw[j].y, raw[j].z, raw[j].w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      v[j][2 * e] = ok ? __uint_as_float(wd[e] << 16) : 0.0f;
      v[j][2 * e + 1] = ok ? __uint_as_float(wd[e] & 0xFFFF0000u) : 0.0f;
    }
    if (has_d) {
      const float dd[8] = {d[j][0].x, d[j][0].y, d[j][0].z, d[j][0].w, d[j][1].x, d[j][1].y, d[j][1].z, d[j][1].w};
#pragma unroll
      for (int e = 0; e < 8; ++e) v[j][e] *= dd[e];
    }
  }

  if constexpr (BITS == 8) {
    // one range per row
    float m = 0.0f;
    if (dynamic) {
#pragma unroll
      for (int j = 0; j < NCH; ++j)
#pragma unroll
        for (int e = 0; e < 8; ++e) m = fmaxf(m, fabsf(v[j][e]));
#pragma unroll
      for (int o = 32; o >= 1; o >>= 1) m = fmaxf(m, __shfl_xor(m, o, 64));
      if constexpr (WPR > 1) {
        __shared__ float red[WPR];
        if (lane == 0) red[wave] = m;
        __syncthreads();
        m = red[0];
#pragma unroll
        for (int w = 1; w < WPR; ++w) m = fmaxf(m, red[w]);
      }
    }
    if (row >= M) return;
    const float delta = (dynamic ? m : cst) / QA;
    float inv = 1.0f / delta;
    if (__builtin_isinf(inv)) inv = 0.0f;
    int8_t* qr = static_cast<int8_t*>(a.qx) + static_cast<size_t>(row) * a.K;
#pragma unroll
    for (int j = 0; j < NCH; ++j) {
      uint32_t b[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        float t = (v[j][e] * g) * inv;
        t = fminf(fmaxf(t, -QA), QA);
        b[e] = rne_code_bits(t);
      }
      const int c = lr + j * LPR;
      if (c < nch)
        *reinterpret_cast<uint2*>(qr + c * 8) =
            make_uint2(pack_low_bytes(b[0], b[1], b[2], b[3]), pack_low_bytes(b[4], b[5], b[6], b[7]));
    }
    if (lr == 0) static_cast<float*>(a.scale)[row] = delta / g;
  } else {
    if (row >= M) return;  // a row's lanes leave together
    uint8_t* qr = static_cast<uint8_t*>(a.qx) + static_cast<size_t>(row) * (F8 ? a.K : a.K / 2);
    uint16_t* sr = static_cast<uint16_t*>(a.scale) + static_cast<size_t>(row) * (a.K / kA4Group);
    float* kr = F8 ? a.kc + static_cast<size_t>(row) * (a.K / kA4Group) : nullptr;
#pragma unroll
    for (int j = 0; j < NCH; ++j) {
      // range of the 64-group: the 8 adjacent lanes holding its chunks
      float m = 0.0f;
      if (dynamic) {
#pragma unroll
        for (int e = 0; e < 8; ++e) m = fmaxf(m, fabsf(v[j][e]));
        m = fmaxf(m, __shfl_xor(m, 1, 64));
        m = fmaxf(m, __shfl_xor(m, 2, 64));
        m = fmaxf(m, __shfl_xor(m, 4, 64));
      }
      const uint32_t dbits = f32_to_f16((dynamic ? m : cst) / QA);
      const float delta = f16_to_f32(dbits);
      float inv = 1.0f / delta;
      if (__builtin_isinf(inv)) inv = 0.0f;
      uint32_t b[8];
      int csum = 0;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        float t = (v[j][e] * g) * inv;
        t = fminf(fmaxf(t, -QA), QA);
        if constexpr (F8) {
          // |code| = rne(|t|) (rounding is symmetric); the sign bit of t
          // becomes the fp8 sign (a code 0 of negative t is -0: value 0)
          const uint32_t m = rne_code_bits(fabsf(t)) & 0xFFu;
          const uint32_t neg = __float_as_uint(t) >> 31;
          b[e] = m | (neg << 7);
          csum += neg ? -static_cast<int>(m) : static_cast<int>(m);
        } else {
          b[e] = rne_code_bits(t);
        }
      }
      const int c = lr + j * LPR;
      if constexpr (F8) {
        // the 64-group's code sum: the 8 adjacent lanes holding its chunks
        csum += __shfl_xor(csum, 1, 64);
        csum += __shfl_xor(csum, 2, 64);
        csum += __shfl_xor(csum, 4, 64);
        if (c < nch) {
          *reinterpret_cast<uint2*>(qr + c * 8) =
              make_uint2(pack_low_bytes(b[0], b[1], b[2], b[3]), pack_low_bytes(b[4], b[5], b[6], b[7]));
          if ((c & 7) == 0) {
            // the fp16 step, widened exactly (an fp32 operand of the fold's fma)
            reinterpret_cast<float*>(a.scale)[static_cast<size_t>(row) * (a.K / kA4Group) + (c >> 3)] = delta;
            // exact: |8 S| < 2^12 and delta has an 11-bit significand
            kr[c >> 3] = (static_cast<float>(-8 * csum) * delta) * 3.814697265625e-06f;  // * 2^-18
          }
        }
      } else {
        // code e < 4 -> low nibble of byte e; code e >= 4 -> high nibble of byte e-4
        const uint32_t lo = pack_low_bytes(b[0], b[1], b[2], b[3]);
        const uint32_t hi = pack_low_bytes(b[4], b[5], b[6], b[7]);
        const uint32_t word = (lo & 0x0F0F0F0Fu) | ((hi << 4) & 0xF0F0F0F0u);
        if (c < nch) {
          *reinterpret_cast<uint32_t*>(qr + c * 4) = word;
          if ((c & 7) == 0) sr[c >> 3] = static_cast<uint16_t>(dbits);
        }
      }
    }
  }
}

template <int BITS, int WPR, int NCH>
hipError_t launch_one(const QuantArgs& a, hipStream_t s) {
  constexpr int RPW = 4 / WPR;
  const dim3 grid = wg_grid((static_cast<size_t>(a.M) + RPW - 1) / RPW);
  if constexpr (BITS == 4) {
    if (a.kc != nullptr) {
      hipLaunchKernelGGL((quantize_act_kernel<BITS, WPR, NCH, true>), grid, dim3(256), 0, s, a);
      return hipGetLastError();
    }
  }
  hipLaunchKernelGGL((quantize_act_kernel<BITS, WPR, NCH, false>), grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

// One wave per row for 8-bit rows of up to 2048 channels when there are many
// rows; otherwise the whole workgroup per row (more lanes per row when rows
// are few or the row is long).
template <int BITS>
hipError_t launch_bits(const QuantArgs& a, hipStream_t s) {
  const int nch = a.K / 8;
  if (BITS == 8 && nch <= 256 && a.M >= 1024) {
    switch ((nch + 63) / 64) {
      case 1: return launch_one<BITS, 1, 1>(a, s);
      case 2: return launch_one<BITS, 1, 2>(a, s);
      case 3: return launch_one<BITS, 1, 3>(a, s);
      case 4: return launch_one<BITS, 1, 4>(a, s);
      default: return hipErrorInvalidValue;
    }
  }
  switch ((nch + 255) / 256) {
    case 1: return launch_one<BITS, 4, 1>(a, s);
    case 2: return launch_one<BITS, 4, 2>(a, s);
    case 3: return launch_one<BITS, 4, 3>(a, s);
    case 4: return launch_one<BITS, 4, 4>(a, s);
    case 5: return launch_one<BITS, 4, 5>(a, s);
    case 6: return launch_one<BITS, 4, 6>(a, s);
    case 7: return launch_one<BITS, 4, 7>(a, s);
    case 8: return launch_one<BITS, 4, 8>(a, s);
    case 9: return launch_one<BITS, 4, 9>(a, s);
    case 10: return launch_one<BITS, 4, 10>(a, s);
    case 11: return launch_one<BITS, 4, 11>(a, s);
    case 12: return launch_one<BITS, 4, 12>(a, s);
    case 13: return launch_one<BITS, 4, 13>(a, s);
    case 14: return launch_one<BITS, 4, 14>(a, s);
    case 15: return launch_one<BITS, 4, 15>(a, s);
    case 16: return launch_one<BITS, 4, 16>(a, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

hipError_t launch_quantize_act(int act_bits, const QuantArgs& a, hipStream_t s) {
  return act_bits == 8 ? launch_bits<8>(a, s) : launch_bits<4>(a, s);
}

}  // namespace sq
