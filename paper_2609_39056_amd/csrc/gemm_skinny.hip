// Weight-streaming GEMM for few tokens (the second fused kernel of Sec. 4.4
// when the layer runs the action and proprioception streams alone): same
// operands, block accumulation and epilogue as the tiled kernel.
#include <algorithm>

#include "gemm_frag.h"
#include "sq_internal.h"

namespace sq {
namespace {

constexpr int TM = 2;  // 32-row MFMA tiles per wave

// Skinny GEMM for few tokens (M <= kSkinnyMaxM; 8-bit activations, one weight
// step per 128 input channels).  The work is streaming the weights.  A
// workgroup owns 64 rows x 32 output channels over a range of K; its four waves
// take alternate stages of that range and keep their own fp32 sums, which are
// added through LDS in wave order at the end.  Operands go straight from
// global memory into registers (the codes of <= 128 tokens stay in L2), one
// stage ahead, so the main loop has no LDS traffic and no barriers.  When the
// output channels alone give too few workgroups, K is also split across
// workgroups: each leaves fp32 sums of its 64 x 32 outputs, which a second
// kernel adds in range order.
constexpr int SK_BM = 64;  // rows per workgroup
constexpr int SK_BN = 32;  // output channels per workgroup

// The operands of one stage for one lane: activation fragments of the two
// 32-row tiles (16 bytes per k-step), the packed weight chunks of the two
// k-step pairs, and the column's fp16 weight step.
struct SkinnyFrag {
  v4i a[TM][4];
  v4u b[2];
  uint32_t w;
};

template <int EPI>
__global__ __launch_bounds__(256, 2) void gemm_skinny_kernel(GemmArgs a) {
  __shared__ float red[3][TM * 16][64];  // sums of waves 1..3
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int M = a.M, N = a.N, K = a.K;
  const int nkt = K / KT;
  const int strips = N / SK_BN;
  const int S = a.split;
  const int strip = blockIdx.x / S, range = blockIdx.x % S;
  const int m0 = blockIdx.y * SK_BM, n0 = strip * SK_BN;
  const int kt0 = range * nkt / S, kt1 = (range + 1) * nkt / S;
  const int h = lane >> 5, col = lane & 31;
  const int rows = min(M - m0, SK_BM);

  // Sources as buffer loads (an optimiser cannot merge those across the
  // loop's two register sets, which would undo the prefetch).  Activation
  // rows past the matrix read the last row; the stage offset goes in the
  // scalar offset.
  const __amdgpu_buffer_rsrc_t rA = buffer_rsrc(static_cast<const int8_t*>(a.qx) + static_cast<size_t>(m0) * K, rows * K);
  const __amdgpu_buffer_rsrc_t rB = buffer_rsrc(a.qw + static_cast<size_t>(n0) * (K / 2), SK_BN * (K / 2));
  const __amdgpu_buffer_rsrc_t rW = buffer_rsrc(a.w_scale + n0, ((nkt - 1) * N + SK_BN) * 2);
  int aoff[TM];
#pragma unroll
  for (int tm = 0; tm < TM; ++tm) aoff[tm] = min(tm * 32 + col, rows - 1) * K + 32 * h;
  const int boff = col * (K / 2) + 16 * h;

  auto load = [&](int kt, SkinnyFrag& f) {
#pragma unroll
    for (int tm = 0; tm < TM; ++tm)
#pragma unroll
      for (int ks = 0; ks < 4; ++ks)
        f.a[tm][ks] = __builtin_bit_cast(
            v4i, __builtin_amdgcn_raw_buffer_load_b128(rA, aoff[tm] + 64 * (ks >> 1) + 16 * (ks & 1), kt * KT, 0));
#pragma unroll
    for (int k2 = 0; k2 < 2; ++k2) f.b[k2] = __builtin_amdgcn_raw_buffer_load_b128(rB, boff + 32 * k2, kt * (KT / 2), 0);
    f.w = __builtin_amdgcn_raw_buffer_load_b16(rW, col * 2, kt * N * 2, 0);  // group-major steps, one group per stage
    __builtin_amdgcn_sched_barrier(0);  // keep the stage's loads ahead of the work after them
  };

  float y[TM][16];
  v16i acc[TM];
#pragma unroll
  for (int tm = 0; tm < TM; ++tm) {
    acc[tm] = (v16i)(0);
#pragma unroll
    for (int r = 0; r < 16; ++r) y[tm][r] = 0.0f;
  }
  float wprev = 0.0f;  // the fold before the first block adds 0

  // y += fp32(C) * Delta_W of the previous block, then this block's MFMAs; a
  // stage that is not this wave's folds with step 0 (adds exactly 0)
  auto compute = [&](const SkinnyFrag& f, bool valid) {
    v4i bf[4];
    bf[0] = unpack_frag(f.b[0][0], f.b[0][1]);
    bf[1] = unpack_frag(f.b[0][2], f.b[0][3]);
    bf[2] = unpack_frag(f.b[1][0], f.b[1][1]);
    bf[3] = unpack_frag(f.b[1][2], f.b[1][3]);
#pragma unroll
    for (int tm = 0; tm < TM; ++tm) {
      fold8(acc[tm], wprev, y[tm]);
      acc[tm] = __builtin_amdgcn_mfma_i32_32x32x32_i8(f.a[tm][0], bf[0], (v16i)(0), 0, 0, 0);
#pragma unroll
      for (int ks = 1; ks < 4; ++ks) acc[tm] = __builtin_amdgcn_mfma_i32_32x32x32_i8(f.a[tm][ks], bf[ks], acc[tm], 0, 0, 0);
    }
    wprev = valid ? f16_to_f32(f.w) * 0.0625f : 0.0f;  // widened weight codes carry a factor 16
  };

  // this wave's stages kt0 + wave + 4j, j < nst, a pair per iteration in two
  // register sets.  The body has no branch, so every load stays ahead of its
  // use: the next stage is always loaded (past the end, the last one again)
  // and each wait leaves one stage of loads in flight.  With nst odd the
  // pair's second stage is a repeat that folds with step 0.
  const int nst = kt1 - kt0 > wave ? (kt1 - kt0 - wave + 3) / 4 : 0;
  auto stage = [&](int j) { return kt0 + wave + 4 * min(j, nst - 1); };
  SkinnyFrag f0, f1;
  if (nst > 0) {
    load(stage(0), f0);
    for (int j = 0; j < nst; j += 2) {
      load(stage(j + 1), f1);
      compute(f0, true);
      load(stage(j + 2), f0);
      compute(f1, j + 1 < nst);
    }
  }
#pragma unroll
  for (int tm = 0; tm < TM; ++tm) fold8(acc[tm], wprev, y[tm]);

  // add the four waves' sums in wave order
  if (wave > 0) {
#pragma unroll
    for (int tm = 0; tm < TM; ++tm)
#pragma unroll
      for (int r = 0; r < 16; ++r) red[wave - 1][tm * 16 + r][lane] = y[tm][r];
  }
  __syncthreads();
  if (wave != 0) return;
#pragma unroll
  for (int w = 0; w < 3; ++w)
#pragma unroll
    for (int tm = 0; tm < TM; ++tm)
#pragma unroll
      for (int r = 0; r < 16; ++r) y[tm][r] += red[w][tm * 16 + r][lane];

  if (S > 1) {
    // this K range's sums, [row][col] of the 64 x 32 block (rows < M)
    float* P = a.partial + (static_cast<size_t>(blockIdx.y * strips + strip) * S + range) * (SK_BM * SK_BN);
#pragma unroll
    for (int tm = 0; tm < TM; ++tm)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = tm * 32 + (r >> 2) * 8 + h * 4 + (r & 3);
        if (m0 + row < M) P[row * SK_BN + col] = y[tm][r];
      }
    return;
  }
  // epilogue: row factor (fetched from the lane that loaded it), bias, cast;
  // a quad transpose gives each lane four consecutive channels of one row
  float rowf = 1.0f, bias = 0.0f;
  if constexpr (EPI == kEpiOut) {
    rowf = static_cast<const float*>(a.act_scale)[min(m0 + lane, M - 1)];
    if (a.bias != nullptr) bias = bf16_to_f32(a.bias[n0 + col]);
  }
  const int rf_bits = __float_as_int(rowf);
  const bool f32out = EPI == kEpiPartial || a.out_dtype == SQ_OUT_F32;
#pragma unroll
  for (int tm = 0; tm < TM; ++tm)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      float v[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int r = g * 4 + q;
        const float rf = __int_as_float(__builtin_amdgcn_ds_bpermute((tm * 32 + g * 8 + h * 4 + q) * 4, rf_bits));
        v[q] = EPI == kEpiPartial ? y[tm][r] : __builtin_fmaf(y[tm][r], rf, bias);
      }
      quad_transpose(v, lane);
      const int m = m0 + tm * 32 + g * 8 + h * 4 + (lane & 3);
      const int n = n0 + (lane & 28);
      if (m < M) {
        if (f32out) {
          *reinterpret_cast<float4*>(static_cast<float*>(a.out) + static_cast<size_t>(m) * N + n) =
              make_float4(v[0], v[1], v[2], v[3]);
        } else {
          uint2 w;
          if (a.out_dtype == SQ_OUT_BF16) {
            const bf16x2 lo = __builtin_convertvector((float2v){v[0], v[1]}, bf16x2);
            const bf16x2 hi = __builtin_convertvector((float2v){v[2], v[3]}, bf16x2);
            w = make_uint2(__builtin_bit_cast(uint32_t, lo), __builtin_bit_cast(uint32_t, hi));
          } else {
            w = make_uint2(f32_to_f16(v[0]) | (f32_to_f16(v[1]) << 16), f32_to_f16(v[2]) | (f32_to_f16(v[3]) << 16));
          }
          *reinterpret_cast<uint2*>(static_cast<uint16_t*>(a.out) + static_cast<size_t>(m) * N + n) = w;
        }
      }
    }
}

// Second kernel of a split skinny GEMM: adds the `split` partial sums of every
// output in range order and finishes it as the skinny epilogue does.  Four
// adjacent outputs per thread.
template <int EPI>
__global__ __launch_bounds__(256) void gemm_skinny_tail_kernel(GemmArgs a) {
  const int strips = a.N / SK_BN;
  const int g = blockIdx.x * 256 + threadIdx.x;  // one thread per 4 outputs of a 64 x 32 block
  const int blk = g / (SK_BM * SK_BN / 4);
  const int e = (g % (SK_BM * SK_BN / 4)) * 4;
  const int row = e / SK_BN, c = e % SK_BN;
  const int mb = blk / strips, strip = blk % strips;
  const int m = mb * SK_BM + row, n = strip * SK_BN + c;
  if (mb * SK_BM >= a.M || m >= a.M) return;
  const float* P = a.partial + static_cast<size_t>(blk) * a.split * (SK_BM * SK_BN) + row * SK_BN + c;
  float4 acc = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
  for (int sl = 0; sl < a.split; ++sl) {
    const float4 v = *reinterpret_cast<const float4*>(P + static_cast<size_t>(sl) * (SK_BM * SK_BN));
    acc.x += v.x;
    acc.y += v.y;
    acc.z += v.z;
    acc.w += v.w;
  }
  float y[4] = {acc.x, acc.y, acc.z, acc.w};
  if constexpr (EPI == kEpiOut) {
    const float rowf = static_cast<const float*>(a.act_scale)[m];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const float b = a.bias != nullptr ? bf16_to_f32(a.bias[n + j]) : 0.0f;
      y[j] = __builtin_fmaf(y[j], rowf, b);
    }
  }
  if (EPI == kEpiPartial || a.out_dtype == SQ_OUT_F32) {
    *reinterpret_cast<float4*>(static_cast<float*>(a.out) + static_cast<size_t>(m) * a.N + n) =
        make_float4(y[0], y[1], y[2], y[3]);
  } else {
    uint2 w;
    if (a.out_dtype == SQ_OUT_BF16) {
      const bf16x2 lo = __builtin_convertvector((float2v){y[0], y[1]}, bf16x2);
      const bf16x2 hi = __builtin_convertvector((float2v){y[2], y[3]}, bf16x2);
      w = make_uint2(__builtin_bit_cast(uint32_t, lo), __builtin_bit_cast(uint32_t, hi));
    } else {
      w = make_uint2(f32_to_f16(y[0]) | (f32_to_f16(y[1]) << 16), f32_to_f16(y[2]) | (f32_to_f16(y[3]) << 16));
    }
    *reinterpret_cast<uint2*>(static_cast<uint16_t*>(a.out) + static_cast<size_t>(m) * a.N + n) = w;
  }
}

}  // namespace

// K ranges per strip of the skinny GEMM: about one workgroup per CU, with at
// least four stages (one per wave) in every range.
static int skinny_split(int32_t M, int32_t N, int32_t K) {
  const int blocks = (N / SK_BN) * ((M + SK_BM - 1) / SK_BM);
  const int nkt = K / KT;
  return std::max(1, std::min(device_cus() / blocks, nkt / 4));
}
size_t skinny_partial_bytes(int32_t M, int32_t N, int32_t K) {
  const int S = skinny_split(M, N, K);
  if (S <= 1) return 0;
  return static_cast<size_t>(N / SK_BN) * ((M + SK_BM - 1) / SK_BM) * S * (SK_BM * SK_BN) * sizeof(float);
}

template <int EPI>
hipError_t launch_skinny_t(const GemmArgs& a0, hipStream_t s, float* partial, size_t partial_bytes) {
  GemmArgs a = a0;
  int S = skinny_split(a.M, a.N, a.K);
  if (S > 1 && (partial == nullptr || partial_bytes < skinny_partial_bytes(a.M, a.N, a.K))) S = 1;
  a.split = S;
  a.partial = S > 1 ? partial : nullptr;
  const int strips = a.N / SK_BN, mblocks = (a.M + SK_BM - 1) / SK_BM;
  hipLaunchKernelGGL((gemm_skinny_kernel<EPI>), dim3(strips * S, mblocks), dim3(256), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || S == 1) return e;
  const int threads = strips * mblocks * (SK_BM * SK_BN / 4);
  hipLaunchKernelGGL((gemm_skinny_tail_kernel<EPI>), dim3((threads + 255) / 256), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_skinny(int epi, const GemmArgs& a, hipStream_t s, float* partial, size_t partial_bytes) {
  switch (epi) {
    case kEpiOut: return launch_skinny_t<kEpiOut>(a, s, partial, partial_bytes);
    case kEpiPartial: return launch_skinny_t<kEpiPartial>(a, s, partial, partial_bytes);
  }
  return hipErrorInvalidValue;
}

}  // namespace sq
