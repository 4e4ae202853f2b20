// Register-level pieces shared by the GEMM kernels: operand types, the int4
// widening of packed fragments, the 8-bit block fold, the quad transpose of
// the register epilogue and raw buffer resources.
#pragma once

#include "sq_internal.h"

namespace sq {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));
typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v16f __attribute__((ext_vector_type(16)));
typedef unsigned int v4u __attribute__((ext_vector_type(4)));
typedef float float2v __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));  // converted with round to nearest even
typedef __attribute__((address_space(3))) uint8_t lds_u8_t;

constexpr int KT = kKTile;   // 128 channels per stage

__device__ __forceinline__ v4i unpack_frag(uint32_t p0, uint32_t p1) {
  uint32_t l0, h0, l1, h1;
  unpack_int4x8_times16(p0, l0, h0);
  unpack_int4x8_times16(p1, l1, h1);
  v4i r;
  r[0] = static_cast<int>(l0);
  r[1] = static_cast<int>(h0);
  r[2] = static_cast<int>(l1);
  r[3] = static_cast<int>(h1);
  return r;
}

// 4 x 4 transpose across the lanes of a quad (lane i = lane & 3): in, lane i
// holds v[q] = element (row q, column i); out, it holds v[j] = element
// (row i, column j).  Two exchanges through DPP quad permutations (VALU only):
// with lane ^ 1 the rows whose low bit differs from the lane's, then with
// lane ^ 2 the column pairs of the row the partner keeps.
__device__ __forceinline__ float dpp_xor1(float x) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), 0xB1, 0xF, 0xF, false));  // quad_perm [1,0,3,2]
}
__device__ __forceinline__ float dpp_xor2(float x) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), 0x4E, 0xF, 0xF, false));  // quad_perm [2,3,0,1]
}
__device__ __forceinline__ void quad_transpose(float (&v)[4], int lane) {
  const bool o1 = lane & 1, o2 = lane & 2;
  // after stage 1 lane i holds rows p, p + 2 (p = i & 1) at columns (i & ~1) + {0, 1}
  const float r0 = dpp_xor1(o1 ? v[0] : v[1]);
  const float r1 = dpp_xor1(o1 ? v[2] : v[3]);
  const float a00 = o1 ? r0 : v[0], a01 = o1 ? v[1] : r0;
  const float a10 = o1 ? r1 : v[2], a11 = o1 ? v[3] : r1;
  // stage 2: lanes with bit 1 clear keep row p, the others row p + 2
  const float u0 = dpp_xor2(o2 ? a00 : a10);
  const float u1 = dpp_xor2(o2 ? a01 : a11);
  v[0] = o2 ? u0 : a00;
  v[1] = o2 ? u1 : a01;
  v[2] = o2 ? a10 : u0;
  v[3] = o2 ? a11 : u1;
}

// y += fp32(C) * Delta_W for one 32 x 32 tile (8-bit activations)
__device__ __forceinline__ void fold8(const v16i& c, float w, float (&yt)[16]) {
#pragma unroll
  for (int r = 0; r < 16; ++r) yt[r] = __builtin_fmaf(static_cast<float>(c[r]), w, yt[r]);
}

// The same fold for an accumulator that started from the integer 0x4B400000
// (the bits of 1.5 * 2^23) instead of 0: for |C| < 2^22 those bits are the
// float 1.5 * 2^23 + C, so one full-rate subtraction gives fp32(C) exactly,
// where v_cvt_f32_i32 issues at about half rate.
constexpr int kMagicAcc = 0x4B400000;
__device__ __forceinline__ void fold8_biased(const v16i& c, float w, float (&yt)[16]) {
#pragma unroll
  for (int r = 0; r < 16; ++r) yt[r] = __builtin_fmaf(__int_as_float(c[r]) - 12582912.0f, w, yt[r]);
}

// The same for the four registers of a 16 x 16 accumulator tile.
__device__ __forceinline__ void fold8_biased4(const v4i& c, float w, float (&yt)[4]) {
#pragma unroll
  for (int r = 0; r < 4; ++r) yt[r] = __builtin_fmaf(__int_as_float(c[r]) - 12582912.0f, w, yt[r]);
}

// LDS byte offset of a __shared__ object.
__device__ __forceinline__ uint32_t lds_offset(const void* p) {
  return static_cast<uint32_t>(reinterpret_cast<uintptr_t>((const lds_u8_t*)p));
}

// One direct global -> LDS load per lane (16 or 4 bytes) from base + voff:
// lane i's data lands at LDS offset `lds` + i * SIZE.  `base` and `lds` must
// be wave-uniform (an SGPR pair and M0); the per-lane part is a 32-bit offset.
// Issued from inline asm so that the compiler, which cannot see which LDS
// bytes such a load writes, does not wait for all of them before every LDS
// read; the kernel waits for them explicitly (wait_vm, wait_vm_and_barrier).  Nothing
// else in these kernels uses M0.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
template <int SIZE>
__device__ __forceinline__ void dma(const void* base, uint32_t voff, uint32_t lds) {
  // readfirstlane returns a signed int: widen through uint32_t (no sign extension)
  const uint64_t b = reinterpret_cast<uint64_t>(base);
  const uint32_t lo = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<int>(static_cast<uint32_t>(b))));
  const uint32_t hi = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<int>(static_cast<uint32_t>(b >> 32))));
  const uint64_t sb = (static_cast<uint64_t>(hi) << 32) | static_cast<uint64_t>(lo);
  const uint32_t m0v = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<int>(lds)));
  if constexpr (SIZE == 16) {
    asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, %2" ::"s"(m0v), "v"(voff), "s"(sb) : "memory", "m0");
  } else {
    static_assert(SIZE == 4, "unsupported size");
    asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dword %1, %2" ::"s"(m0v), "v"(voff), "s"(sb) : "memory", "m0");
  }
}
#pragma clang diagnostic pop

// Wait until at most N of this wave's vector-memory operations are in flight
// (the wave's own direct loads; no workgroup barrier).
template <int N>
__device__ __forceinline__ void wait_vm() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// fp32(C) * sigma for the fp16 step in half HI of `pair` (4-bit activation
// group steps, two per dword): one v_fma_mix_f32 converts the half and
// multiplies with one rounding, the same value as the conversion followed by
// an fp32 multiply.
typedef _Float16 half2v __attribute__((ext_vector_type(2)));
template <int HI>
__device__ __forceinline__ float mul_step16(float cf, uint32_t pair) {
  return __builtin_fmaf(cf, static_cast<float>(__builtin_bit_cast(half2v, pair)[HI]), 0.0f);
}

// The sums of four adjacent outputs over the S ranges of a split K, range r
// at P + r * stride (16-byte aligned), added in range order: fp32, or with
// INT the raw bits of int32 sums (one weight step per channel).  The loads go
// out eight at a time before any addition (a slot past S re-reads the last
// range and is not added), so the sum waits about one memory latency per
// eight ranges instead of one per range; the additions and their order are
// those of a plain loop over r.
template <bool INT>
__device__ __forceinline__ float4 sum_ranges4(const float* P, size_t stride, int S) {
  float4 f = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
  int4 q = make_int4(0, 0, 0, 0);
  for (int s0 = 0; s0 < S; s0 += 8) {
    float4 v[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] = *reinterpret_cast<const float4*>(P + static_cast<size_t>(min(s0 + i, S - 1)) * stride);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      if (s0 + i < S) {
        if constexpr (INT) {
          q.x += __float_as_int(v[i].x);
          q.y += __float_as_int(v[i].y);
          q.z += __float_as_int(v[i].z);
          q.w += __float_as_int(v[i].w);
        } else {
          f.x += v[i].x;
          f.y += v[i].y;
          f.z += v[i].z;
          f.w += v[i].w;
        }
      }
    }
  }
  if constexpr (INT) return make_float4(__int_as_float(q.x), __int_as_float(q.y), __int_as_float(q.z), __int_as_float(q.w));
  return f;
}

// Word 3 of a raw buffer resource (32-bit data format, no swizzle).
constexpr int kBufWord3 = 0x00020000;

// Raw buffer resource over [base, base + bytes): loads past the end return 0.
template <typename T>
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_rsrc(const T* base, int bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<T*>(base), 0, bytes, kBufWord3);
}

}  // namespace
}  // namespace sq
