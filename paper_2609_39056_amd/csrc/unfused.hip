// The unfused execution that Rudder's fusion removes (Sec. 4.4: executing
// channel scaling, stream gains and output compensation separately adds
// launches and intermediate traffic).  Each stage is its own kernel and hands
// an fp32 (or int32) tensor to the next through HBM:
//
//   U1  x~ = X D^-1              -> fp32 [M][K], plus the amax of each row
//                                   (8-bit) or 64-group (4-bit)
//   U2  x^ = x~ * gamma_s(i)     -> fp32 [M][K]
//   U3  q  = Q(x^; Delta)        -> codes, Delta (fp32 [M]) or sigma (fp16)
//   U4  GEMM                     -> int32 C [M][N] (8-bit, one weight step per
//                                   output channel) or the fp32 block sum
//                                   sum_b fp32(C^b) s_b Delta_W  [M][N]
//   U5  dequantize (x Delta_X, and x Delta_W for int32 C)   -> fp32 [M][N]
//   U6  inverse-gain compensation (x 1/gamma_s(i))          -> fp32 [M][N]
//   U7  + bias, cast                                        -> y
//
// The codes come out bit-identical to the fused path (same fp32 operations in
// the same order: (x~ * g) * inv), so only the fp32 rounding of the epilogue
// differs.
#include "sq_internal.h"

namespace sq {
namespace {

// U1: one workgroup per row.
__global__ __launch_bounds__(256) void u1_scale_kernel(UnfusedArgs a) {
  const size_t wg = flat_wg();
  if (wg >= static_cast<size_t>(a.M)) return;  // the whole workgroup: before any barrier
  const int row = static_cast<int>(wg);
  const int tid = threadIdx.x;
  const int nch = a.K / 8;
  const uint16_t* xr = a.x + static_cast<size_t>(row) * a.K;
  float* xo = a.xt + static_cast<size_t>(row) * a.K;
  float rmax = 0.0f;
  for (int c = tid; c < nch; c += 256) {
    const uint4 raw = *reinterpret_cast<const uint4*>(xr + c * 8);
    const uint32_t wd[4] = {raw.x, raw.y, raw.z, raw.w};
    float v[8];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      v[2 * e] = __uint_as_float(wd[e] << 16);
      v[2 * e + 1] = __uint_as_float(wd[e] & 0xFFFF0000u);
    }
    if (a.dinv != nullptr) {
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] *= a.dinv[c * 8 + e];
    }
    *reinterpret_cast<float4*>(xo + c * 8) = make_float4(v[0], v[1], v[2], v[3]);
    *reinterpret_cast<float4*>(xo + c * 8 + 4) = make_float4(v[4], v[5], v[6], v[7]);
    float m = 0.0f;
#pragma unroll
    for (int e = 0; e < 8; ++e) m = fmaxf(m, fabsf(v[e]));
    if (a.act_bits == 4) {
      m = fmaxf(m, __shfl_xor(m, 1, 64));
      m = fmaxf(m, __shfl_xor(m, 2, 64));
      m = fmaxf(m, __shfl_xor(m, 4, 64));
      if ((c & 7) == 0) a.gmax[static_cast<size_t>(row) * (a.K / kA4Group) + (c >> 3)] = m;
    } else {
      rmax = fmaxf(rmax, m);
    }
  }
  if (a.act_bits == 8) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) rmax = fmaxf(rmax, __shfl_xor(rmax, o, 64));
    __shared__ float red[4];
    if ((tid & 63) == 0) red[tid >> 6] = rmax;
    __syncthreads();
    if (tid == 0) a.gmax[row] = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  }
}

// U2: elementwise gain.
__global__ __launch_bounds__(256) void u2_gain_kernel(UnfusedArgs a) {
  const size_t n4 = static_cast<size_t>(a.M) * a.K / 4;
  for (size_t i = blockIdx.x * 256ull + threadIdx.x; i < n4; i += static_cast<size_t>(gridDim.x) * 256) {
    const int row = static_cast<int>((i * 4) / a.K);
    const float g = a.gamma[a.step * a.S + a.tok2stream[row]];
    float4 v = reinterpret_cast<const float4*>(a.xt)[i];
    v.x *= g; v.y *= g; v.z *= g; v.w *= g;
    reinterpret_cast<float4*>(a.xh)[i] = v;
  }
}

// U3: quantize x^ with the step of its row / group; one thread per 8-chunk.
__global__ __launch_bounds__(256) void u3_quant_kernel(UnfusedArgs a) {
  const int nch = a.K / 8;
  const size_t total = static_cast<size_t>(a.M) * nch;
  const float QA = a.act_bits == 8 ? 127.0f : 7.0f;
  for (size_t i = blockIdx.x * 256ull + threadIdx.x; i < total; i += static_cast<size_t>(gridDim.x) * 256) {
    const int row = static_cast<int>(i / nch);
    const int c = static_cast<int>(i % nch);
    float cr;
    if (a.range_mode == SQ_RANGE_STATIC) {
      cr = a.clip[a.step];
    } else {
      cr = a.act_bits == 8 ? a.gmax[row] : a.gmax[static_cast<size_t>(row) * (a.K / kA4Group) + (c >> 3)];
    }
    float delta = cr / QA;
    uint32_t dbits = 0;
    if (a.act_bits == 4) {
      dbits = f32_to_f16(delta);
      delta = f16_to_f32(dbits);
    }
    float inv = 1.0f / delta;
    if (__builtin_isinf(inv)) inv = 0.0f;
    const float* xr = a.xh + static_cast<size_t>(row) * a.K + c * 8;
    int q[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      float t = xr[e] * inv;
      t = fminf(fmaxf(t, -QA), QA);
      q[e] = static_cast<int>(__builtin_rintf(t));
    }
    if (a.act_bits == 8) {
      uint32_t w0 = 0, w1 = 0;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        w0 |= (static_cast<uint32_t>(q[e]) & 0xFFu) << (8 * e);
        w1 |= (static_cast<uint32_t>(q[e + 4]) & 0xFFu) << (8 * e);
      }
      *reinterpret_cast<uint2*>(static_cast<int8_t*>(a.qx) + static_cast<size_t>(row) * a.K + c * 8) =
          make_uint2(w0, w1);
      if (c == 0) static_cast<float*>(a.qscale)[row] = delta;
    } else {
      uint32_t w = 0;
#pragma unroll
      for (int e = 0; e < 8; ++e)
        w |= (static_cast<uint32_t>(q[e]) & 0xFu) << (8 * (e & 3) + 4 * (e >> 2));
      *reinterpret_cast<uint32_t*>(static_cast<uint8_t*>(a.qx) + static_cast<size_t>(row) * (a.K / 2) + c * 4) = w;
      if ((c & 7) == 0)
        static_cast<uint16_t*>(a.qscale)[static_cast<size_t>(row) * (a.K / kA4Group) + (c >> 3)] =
            static_cast<uint16_t>(dbits);
    }
  }
}

// U5: activation step (8-bit).  int32 C: (fp32(C) * Delta_X) * Delta_W[j];
// fp32 block sum: P * Delta_X.
__global__ __launch_bounds__(256) void u5_dequant_kernel(UnfusedArgs a) {
  const size_t total = static_cast<size_t>(a.M) * a.N;
  const bool int_c = a.w_group == a.K;
  for (size_t i = blockIdx.x * 256ull + threadIdx.x; i < total; i += static_cast<size_t>(gridDim.x) * 256) {
    const int row = static_cast<int>(i / a.N);
    const int col = static_cast<int>(i % a.N);
    const float dx = static_cast<const float*>(a.qscale)[row];
    float v;
    if (int_c) {
      // one weight group spanning K: the group-major steps are w_scale[col]
      v = (static_cast<float>(static_cast<const int32_t*>(a.gemm_out)[i]) * dx) * f16_to_f32(a.w_scale[col]);
    } else {
      v = static_cast<const float*>(a.gemm_out)[i] * dx;
    }
    a.y1[i] = v;
  }
}

// U6: inverse-gain output compensation.
__global__ __launch_bounds__(256) void u6_comp_kernel(UnfusedArgs a, const float* src) {
  const size_t total = static_cast<size_t>(a.M) * a.N;
  for (size_t i = blockIdx.x * 256ull + threadIdx.x; i < total; i += static_cast<size_t>(gridDim.x) * 256) {
    const int row = static_cast<int>(i / a.N);
    const float kappa = 1.0f / a.gamma[a.step * a.S + a.tok2stream[row]];
    a.y2[i] = src[i] * kappa;
  }
}

// U7: bias and cast.
__global__ __launch_bounds__(256) void u7_bias_cast_kernel(UnfusedArgs a) {
  const size_t total = static_cast<size_t>(a.M) * a.N;
  for (size_t i = blockIdx.x * 256ull + threadIdx.x; i < total; i += static_cast<size_t>(gridDim.x) * 256) {
    const int col = static_cast<int>(i % a.N);
    float v = a.y2[i];
    if (a.bias != nullptr) v = v + bf16_to_f32(a.bias[col]);
    if (a.out_dtype == SQ_OUT_F32) {
      static_cast<float*>(a.y)[i] = v;
    } else if (a.out_dtype == SQ_OUT_BF16) {
      static_cast<uint16_t*>(a.y)[i] = static_cast<uint16_t>(f32_to_bf16(v));
    } else {
      static_cast<uint16_t*>(a.y)[i] = static_cast<uint16_t>(f32_to_f16(v));
    }
  }
}

unsigned grid_for(size_t n) {
  size_t g = (n + 255) / 256;
  return static_cast<unsigned>(g < 8192 ? (g == 0 ? 1 : g) : 8192);
}

}  // namespace

hipError_t launch_unfused(const UnfusedArgs& a, hipStream_t s) {
  hipError_t e;
  hipLaunchKernelGGL(u1_scale_kernel, wg_grid(static_cast<size_t>(a.M)), dim3(256), 0, s, a);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL(u2_gain_kernel, dim3(grid_for(static_cast<size_t>(a.M) * a.K / 4)), dim3(256), 0, s, a);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL(u3_quant_kernel, dim3(grid_for(static_cast<size_t>(a.M) * a.K / 8)), dim3(256), 0, s, a);
  if ((e = hipGetLastError()) != hipSuccess) return e;

  // U4: the same int8-MFMA main loop as the fused path, writing its
  // accumulators (int32) or block sums (fp32) to memory instead of finishing.
  GemmArgs g{};
  g.qx = a.qx;
  g.act_scale = a.qscale;
  g.tok2stream = a.tok2stream;
  g.gamma = a.gamma;
  g.S = a.S;
  g.step = a.step;
  g.qw = a.qw;
  g.w_scale = a.w_scale;
  g.bias = nullptr;
  g.out = a.gemm_out;
  g.M = a.M;
  g.N = a.N;
  g.K = a.K;
  g.w_group = a.w_group;
  g.out_dtype = SQ_OUT_F32;
  const bool int_c = a.act_bits == 8 && a.w_group == a.K;
  e = launch_gemm(a.act_bits, int_c ? kEpiInt32 : kEpiPartial, g, s);
  if (e != hipSuccess) return e;

  const size_t mn = static_cast<size_t>(a.M) * a.N;
  const float* comp_src = a.y1;
  if (a.act_bits == 8) {
    hipLaunchKernelGGL(u5_dequant_kernel, dim3(grid_for(mn)), dim3(256), 0, s, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  } else {
    comp_src = static_cast<const float*>(a.gemm_out);  // 4-bit: sigma and Delta_W applied in U4
  }
  hipLaunchKernelGGL(u6_comp_kernel, dim3(grid_for(mn)), dim3(256), 0, s, a, comp_src);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL(u7_bias_cast_kernel, dim3(grid_for(mn)), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace sq
