// The second fused kernel of Sec. 4.4: Q_X Q_W with int32 accumulation on the
// gfx950 int8 matrix cores, and the dequantization epilogue of Eq. 10 in
// registers.  The int32 products and scaled activations never reach memory.
//
// Operands.  gfx950 has no int4 integer MFMA, so int4 codes are widened to
// int8: a packed dword holding codes k0..k7 (k_b low nibble, k_{b+4} high
// nibble of byte b) becomes two int8 dwords by a shift and a mask, each byte
// being 16 * code.  The int32 result is then 16 * C (weights) or 256 * C
// (4-bit weights and 4-bit activations); the power-of-two factor is folded
// exactly into the fp32 scale (no rounding changes, no overflow: |C| < 2^27).
//
// Tiling.  A 256-thread workgroup computes a 128 x 128 output tile; its four
// waves each own 64 x 64 = 2 x 2 tiles of v_mfma_i32_32x32x32_i8.  K advances
// in stages of 128: the activation tile (int8 or packed int4) and the packed
// weight tile are copied global -> registers -> LDS (double-buffered, one
// barrier per stage) with 16-byte coalesced loads; waves read MFMA fragments
// from LDS with row pitches chosen so that the 16-byte (8-bit) and 8-byte
// (packed) fragment reads are free of bank conflicts.
//
// Dequantization.  One int32 accumulator per K-block (the weight group for
// 8-bit activations, 64 for 4-bit).  At the end of a block each accumulator is
// converted and folded into an fp32 sum: y += fp32(C) * Delta_W (8-bit; the
// row scale r_i factors out and is applied once in the epilogue) or
// y += (fp32(C) * sigma_i) * Delta_W (4-bit).  The epilogue multiplies by r_i
// (8-bit) or kappa_i = 1/gamma (4-bit), adds the bias and casts.
#include "sq_internal.h"

namespace sq {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));

constexpr int BM = 128;
constexpr int BN = 128;
constexpr int KT = kKTile;            // 128
constexpr int TM = 2;                 // 32-row MFMA tiles per wave
constexpr int TN = 2;                 // 32-col MFMA tiles per wave
constexpr int GROUP_M = 8;            // m-tiles per supertile (L2 reuse)

__device__ __forceinline__ v4i unpack_frag(uint2 p) {
  uint32_t l0, h0, l1, h1;
  unpack_int4x8_times16(p.x, l0, h0);
  unpack_int4x8_times16(p.y, l1, h1);
  v4i r;
  r[0] = static_cast<int>(l0);
  r[1] = static_cast<int>(h0);
  r[2] = static_cast<int>(l1);
  r[3] = static_cast<int>(h1);
  return r;
}

// Workgroup -> output tile.  Workgroups are dealt to the 8 XCDs round-robin;
// renumber them so each XCD runs a contiguous range of logical tiles, then walk
// the logical range in supertiles of GROUP_M m-tiles so that tiles running at
// the same time on one XCD share activation rows and weight columns in its L2.
__device__ __forceinline__ void tile_of(int ntm, int ntn, int& tm, int& tn) {
  const int nblk = gridDim.x;
  const int bid = blockIdx.x;
  const int q = nblk / 8, r = nblk % 8;
  const int xcd = bid % 8, i = bid / 8;
  const int lid = xcd * q + min(xcd, r) + i;
  const int per_group = GROUP_M * ntn;
  const int group = lid / per_group;
  const int first_m = group * GROUP_M;
  const int gm = min(ntm - first_m, GROUP_M);
  const int in_group = lid % per_group;
  tm = first_m + in_group % gm;
  tn = in_group / gm;
}

// Write int32 block accumulators (test hook / unfused int32 path); the
// widened codes carry a factor 16 (weights) or 256 (both operands 4-bit).
template <int ABITS>
__device__ __forceinline__ void dump_block(const GemmArgs& a, const v16i (&acc)[TM][TN], int blk, int m0,
                                           int n0, int wm, int wn, int lane) {
  int32_t* out = static_cast<int32_t*>(a.out);
  constexpr int SHIFT = ABITS == 8 ? 4 : 8;
#pragma unroll
  for (int tm = 0; tm < TM; ++tm)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int m = m0 + wm * 64 + tm * 32 + (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3);
      if (m >= a.M) continue;
#pragma unroll
      for (int tn = 0; tn < TN; ++tn) {
        const int n = n0 + wn * 64 + tn * 32 + (lane & 31);
        if (n < a.N) out[(static_cast<size_t>(blk) * a.M + m) * a.N + n] = acc[tm][tn][r] >> SHIFT;
      }
    }
}

typedef __attribute__((address_space(3))) uint8_t lds_u8_t;

// LDS byte offset of a __shared__ object.
__device__ __forceinline__ uint32_t lds_offset(const void* p) {
  return static_cast<uint32_t>(reinterpret_cast<uintptr_t>((const lds_u8_t*)p));
}

// One direct global -> LDS load per lane (16 or 4 bytes): lane i's data lands
// at LDS offset `lds` + i * SIZE; `lds` must be wave-uniform (it goes to M0).
// Issued from inline asm so that the compiler, which cannot see which LDS
// bytes such a load writes, does not wait for all of them before every LDS
// read; the kernel waits for them explicitly (wait_vm_and_barrier).  Nothing
// else in these kernels uses M0.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
template <int SIZE>
__device__ __forceinline__ void dma(const void* src, uint32_t lds) {
  const uint32_t m0v = __builtin_amdgcn_readfirstlane(lds);
  if constexpr (SIZE == 16) {
    asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, off" ::"s"(m0v), "v"(src) : "memory", "m0");
  } else {
    static_assert(SIZE == 4, "unsupported size");
    asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dword %1, off" ::"s"(m0v), "v"(src) : "memory", "m0");
  }
}
#pragma clang diagnostic pop

// Wait until at most N of this wave's vector-memory operations are in flight,
// then synchronize the workgroup.  One asm block with a memory clobber: no LDS
// access moves across it (a fenced __syncthreads would instead drain every
// outstanding load, including the stages still in flight).
template <int N>
__device__ __forceinline__ void wait_vm_and_barrier() {
  asm volatile("s_waitcnt vmcnt(%0)\n\ts_barrier" ::"n"(N) : "memory");
}

// LDS layout of one pipeline stage (no padding; 16-byte chunks XOR-swizzled
// so that the fragment reads of 16 consecutive rows hit 16 distinct bank
// groups):
//   8-bit activations: row r (128 B) holds chunk c at position c ^ ((r >> 1) & 7)
//   packed int4 rows (weights, 4-bit activations; 64 B): c at c ^ ((r >> 2) & 3)
//   4-bit group steps: the two fp16 steps of row r in the dword at
//     (r / 32) * 256 + (r % 32) * 4 (wave w loads rows 32w..32w+31, twice)
//   weight steps: wave w, lane i -> the aligned dword holding the fp16 step of
//     output channel wn * 64 + i, at w * 256 + i * 4
// Lane (row, h = lane >> 5) feeds MFMA k-step s (0..3) of a stage with the
// channels [64 (s >> 1) + 32 h + 16 (s & 1), +16): for 8-bit activations the
// 16-byte chunk 4 (s >> 1) + 2 h + (s & 1); for packed rows the low (s even)
// or high (s odd) half of chunk 2 (s >> 1) + h, so one 16-byte read serves two
// k-steps.  Activations and weights use the same assignment, so every product
// pairs equal channels, and k-steps {0, 1} cover channels [0, 64), {2, 3}
// cover [64, 128): a 64-wide block never straddles an MFMA.
template <int ABITS>
struct Layout {
  static constexpr int A_BYTES = ABITS == 8 ? BM * KT : BM * KT / 2;
  static constexpr int B_BYTES = BN * KT / 2;
  static constexpr int S_BYTES = ABITS == 4 ? 4 * 256 : 0;
  static constexpr int W_BYTES = 4 * 256;
  static constexpr int STAGE = A_BYTES + B_BYTES + S_BYTES + W_BYTES;
};
constexpr int STAGES = 3;

// ABITS: 8 or 4.  EPI: EpiMode.  W128: 8-bit activations with one weight step
// per 128 input channels (one K-block per pipeline stage); otherwise a block
// spans w_group / 128 stages (8-bit) or half a stage (4-bit).
template <int ABITS, int EPI, bool W128>
__global__ __launch_bounds__(256, 2) void gemm_w4_kernel(GemmArgs a) {
  using LY = Layout<ABITS>;
  constexpr bool NEED_SCALE = (EPI == kEpiOut || EPI == kEpiPartial);
  constexpr bool LOAD_SIGMA = ABITS == 4 && NEED_SCALE;
  // direct loads per wave per stage: activations, weights, group steps, weight steps
  constexpr int NDMA = (ABITS == 8 ? 4 : 2) + 2 + (LOAD_SIGMA ? 1 : 0) + (NEED_SCALE ? 1 : 0);

  __shared__ __align__(1024) uint8_t smem[STAGES * LY::STAGE];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int h = lane >> 5;
  const int M = a.M, N = a.N, K = a.K;

  const int ntm = (M + BM - 1) / BM;
  const int ntn = (N + BN - 1) / BN;
  int tile_m, tile_n;
  tile_of(ntm, ntn, tile_m, tile_n);
  const int m0 = tile_m * BM;
  const int n0 = tile_n * BN;
  const int nkt = K / KT;
  const int nwg = K / a.w_group;
  const uint8_t* qx = static_cast<const uint8_t*>(a.qx);
  const uint32_t smem_lds = lds_offset(smem);

  // ---- per-lane global sources of this wave's direct loads (stage 0)
  const uint8_t* srcA[ABITS == 8 ? 4 : 2];
  const uint8_t* srcB[2];
  const uint8_t* srcS = nullptr;
  const uint8_t* srcW = nullptr;
  if constexpr (ABITS == 8) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = 8 * (4 * wave + i) + (lane >> 3);
      const int c = (lane & 7) ^ ((row >> 1) & 7);
      srcA[i] = qx + static_cast<size_t>(min(m0 + row, M - 1)) * K + c * 16;
    }
  } else {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int row = 16 * (2 * wave + i) + (lane >> 2);
      const int c = (lane & 3) ^ ((row >> 2) & 3);
      srcA[i] = qx + static_cast<size_t>(min(m0 + row, M - 1)) * (K / 2) + c * 16;
    }
  }
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int col = 16 * (2 * wave + i) + (lane >> 2);
    const int c = (lane & 3) ^ ((col >> 2) & 3);
    srcB[i] = a.qw + static_cast<size_t>(min(n0 + col, N - 1)) * (K / 2) + c * 16;
  }
  if constexpr (LOAD_SIGMA) {
    const int row = 32 * wave + (lane & 31);
    srcS = static_cast<const uint8_t*>(a.act_scale) + static_cast<size_t>(min(m0 + row, M - 1)) * (K / kA4Group) * 2;
  }
  // weight steps: element (column, group) sits in the dword at element index
  // & ~1 (the array has an even number of elements: N % 64 == 0)
  const int wcol = min(n0 + wn * 64 + lane, N - 1);
  if constexpr (NEED_SCALE) srcW = reinterpret_cast<const uint8_t*>(a.w_scale);

  auto issue_stage = [&](int kt) {
    const uint32_t st = smem_lds + (kt % STAGES) * LY::STAGE;
    if constexpr (ABITS == 8) {
#pragma unroll
      for (int i = 0; i < 4; ++i) dma<16>(srcA[i] + kt * KT, st + (4 * wave + i) * 1024);
    } else {
#pragma unroll
      for (int i = 0; i < 2; ++i) dma<16>(srcA[i] + kt * (KT / 2), st + (2 * wave + i) * 1024);
    }
#pragma unroll
    for (int i = 0; i < 2; ++i) dma<16>(srcB[i] + kt * (KT / 2), st + LY::A_BYTES + (2 * wave + i) * 1024);
    if constexpr (LOAD_SIGMA) dma<4>(srcS + kt * 4, st + LY::A_BYTES + LY::B_BYTES + wave * 256);
    if constexpr (NEED_SCALE) {
      const size_t e = static_cast<size_t>(wcol) * nwg + (kt * KT) / a.w_group;
      dma<4>(srcW + (e & ~static_cast<size_t>(1)) * 2, st + LY::A_BYTES + LY::B_BYTES + LY::S_BYTES + wave * 256);
    }
  };

  v16i acc[TM][TN];
  float y[TM][TN][16];
#pragma unroll
  for (int tm = 0; tm < TM; ++tm)
#pragma unroll
    for (int tn = 0; tn < TN; ++tn) {
      acc[tm][tn] = (v16i)(0);
#pragma unroll
      for (int r = 0; r < 16; ++r) y[tm][tn][r] = 0.0f;
    }

  issue_stage(0);
  if (nkt > 1) {
    issue_stage(1);
    wait_vm_and_barrier<NDMA>();
  } else {
    wait_vm_and_barrier<0>();
  }

  for (int kt = 0; kt < nkt; ++kt) {
    const bool pre = kt + 2 < nkt;
    if (pre) issue_stage(kt + 2);

    if constexpr (ABITS == 8 && !W128) {
      if ((kt * KT) % a.w_group == 0) {
#pragma unroll
        for (int tm = 0; tm < TM; ++tm)
#pragma unroll
          for (int tn = 0; tn < TN; ++tn) acc[tm][tn] = (v16i)(0);
      }
    }

    const uint8_t* A = smem + (kt % STAGES) * LY::STAGE;
    const uint8_t* B = A + LY::A_BYTES;
    const uint8_t* S = B + LY::B_BYTES;
    const uint32_t* Wst = reinterpret_cast<const uint32_t*>(S + LY::S_BYTES + wave * 256);

    // Weight steps of this stage for the owned columns (one per 32-wide
    // tile); the 1/16 (8-bit) or 1/256 (4-bit) of the widened codes is folded in.
    float wsv[TN];
    if constexpr (NEED_SCALE) {
      const int wb = (kt * KT) / a.w_group;
#pragma unroll
      for (int tn = 0; tn < TN; ++tn) {
        const int col = min(n0 + wn * 64 + tn * 32 + (lane & 31), N - 1);
        const uint32_t pair = Wst[tn * 32 + (lane & 31)];
        const uint32_t bits = ((static_cast<size_t>(col) * nwg + wb) & 1) ? (pair >> 16) : (pair & 0xFFFFu);
        wsv[tn] = f16_to_f32(bits) * (ABITS == 8 ? 0.0625f : 0.00390625f);
      }
    }

    uint4 pa[TM], pb[TN];
#pragma unroll
    for (int ks = 0; ks < KT / 32; ++ks) {
      v4i af[TM], bf[TN];
#pragma unroll
      for (int tm = 0; tm < TM; ++tm) {
        const int row = wm * 64 + tm * 32 + (lane & 31);
        if constexpr (ABITS == 8) {
          const int c = (4 * (ks >> 1) + 2 * h + (ks & 1)) ^ ((row >> 1) & 7);
          af[tm] = *reinterpret_cast<const v4i*>(A + row * KT + c * 16);
        } else {
          if ((ks & 1) == 0) {
            const int c = (2 * (ks >> 1) + h) ^ ((row >> 2) & 3);
            pa[tm] = *reinterpret_cast<const uint4*>(A + row * (KT / 2) + c * 16);
          }
          af[tm] = (ks & 1) ? unpack_frag(make_uint2(pa[tm].z, pa[tm].w)) : unpack_frag(make_uint2(pa[tm].x, pa[tm].y));
        }
      }
#pragma unroll
      for (int tn = 0; tn < TN; ++tn) {
        if ((ks & 1) == 0) {
          const int col = wn * 64 + tn * 32 + (lane & 31);
          const int c = (2 * (ks >> 1) + h) ^ ((col >> 2) & 3);
          pb[tn] = *reinterpret_cast<const uint4*>(B + col * (KT / 2) + c * 16);
        }
        bf[tn] = (ks & 1) ? unpack_frag(make_uint2(pb[tn].z, pb[tn].w)) : unpack_frag(make_uint2(pb[tn].x, pb[tn].y));
      }
      // A block starts here: at every stage (8-bit, 128-wide weight groups)
      // or every 64 channels (4-bit); a zero accumulator input costs nothing.
      const bool zero_c = ABITS == 8 ? (W128 && ks == 0) : ((ks & 1) == 0);
#pragma unroll
      for (int tm = 0; tm < TM; ++tm)
#pragma unroll
        for (int tn = 0; tn < TN; ++tn) {
          if (zero_c)
            acc[tm][tn] = __builtin_amdgcn_mfma_i32_32x32x32_i8(af[tm], bf[tn], (v16i)(0), 0, 0, 0);
          else
            acc[tm][tn] = __builtin_amdgcn_mfma_i32_32x32x32_i8(af[tm], bf[tn], acc[tm][tn], 0, 0, 0);
        }

      if constexpr (ABITS == 4) {
        if ((ks & 1) == 1) {  // end of a 64-wide block
          const int hb = ks >> 1;
          if constexpr (EPI == kEpiDump) {
            dump_block<ABITS>(a, acc, kt * 2 + hb, m0, n0, wm, wn, lane);
          } else {
#pragma unroll
            for (int tm = 0; tm < TM; ++tm)
#pragma unroll
              for (int r4 = 0; r4 < 4; ++r4) {
                const int ml = wm * 64 + tm * 32 + r4 * 8 + (lane >> 5) * 4;
                // four rows x two fp16 steps; this block's step is the hb-th
                const uint4 sp = *reinterpret_cast<const uint4*>(S + (ml >> 5) * 256 + (ml & 31) * 4);
                const uint32_t w4[4] = {sp.x, sp.y, sp.z, sp.w};
#pragma unroll
                for (int tn = 0; tn < TN; ++tn)
#pragma unroll
                  for (int i = 0; i < 4; ++i) {
                    const int r = r4 * 4 + i;
                    const float sg = f16_to_f32(hb ? (w4[i] >> 16) : (w4[i] & 0xFFFFu));
                    const float t = static_cast<float>(acc[tm][tn][r]) * sg;
                    y[tm][tn][r] = __builtin_fmaf(t, wsv[tn], y[tm][tn][r]);
                  }
              }
          }
        }
      }
    }

    if constexpr (ABITS == 8) {
      if (W128 || ((kt + 1) * KT) % a.w_group == 0) {  // end of a weight group
        if constexpr (EPI == kEpiDump) {
          dump_block<ABITS>(a, acc, ((kt + 1) * KT) / a.w_group - 1, m0, n0, wm, wn, lane);
        } else if constexpr (EPI != kEpiInt32) {
#pragma unroll
          for (int tm = 0; tm < TM; ++tm)
#pragma unroll
            for (int tn = 0; tn < TN; ++tn)
#pragma unroll
              for (int r = 0; r < 16; ++r)
                y[tm][tn][r] = __builtin_fmaf(static_cast<float>(acc[tm][tn][r]), wsv[tn], y[tm][tn][r]);
        }
      }
    }

    if (pre) {
      wait_vm_and_barrier<NDMA>();
    } else {
      wait_vm_and_barrier<0>();
    }
  }

  if constexpr (EPI == kEpiInt32) {
    dump_block<ABITS>(a, acc, 0, m0, n0, wm, wn, lane);
    return;
  }
  if constexpr (EPI == kEpiDump) return;

  // Epilogue: row factor, bias, cast, store.
#pragma unroll
  for (int tm = 0; tm < TM; ++tm)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int m = m0 + wm * 64 + tm * 32 + (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3);
      if (m >= M) continue;
      float rowf = 1.0f;
      if constexpr (EPI == kEpiOut) {
        if constexpr (ABITS == 8) {
          rowf = static_cast<const float*>(a.act_scale)[m];
        } else {
          rowf = 1.0f / a.gamma[a.step * a.S + a.tok2stream[m]];
        }
      }
#pragma unroll
      for (int tn = 0; tn < TN; ++tn) {
        const int n = n0 + wn * 64 + tn * 32 + (lane & 31);
        if (n >= N) continue;
        const size_t o = static_cast<size_t>(m) * N + n;
        if constexpr (EPI == kEpiPartial) {
          static_cast<float*>(a.out)[o] = y[tm][tn][r];
        } else {
          const float b = a.bias != nullptr ? bf16_to_f32(a.bias[n]) : 0.0f;
          const float v = __builtin_fmaf(y[tm][tn][r], rowf, b);
          if (a.out_dtype == SQ_OUT_F32) {
            static_cast<float*>(a.out)[o] = v;
          } else if (a.out_dtype == SQ_OUT_BF16) {
            static_cast<uint16_t*>(a.out)[o] = static_cast<uint16_t>(f32_to_bf16(v));
          } else {
            static_cast<uint16_t*>(a.out)[o] = static_cast<uint16_t>(f32_to_f16(v));
          }
        }
      }
    }
}

template <int ABITS, int EPI, bool W128>
hipError_t launch_t(const GemmArgs& a, hipStream_t s) {
  const unsigned grid = static_cast<unsigned>(((a.M + BM - 1) / BM) * ((a.N + BN - 1) / BN));
  hipLaunchKernelGGL((gemm_w4_kernel<ABITS, EPI, W128>), dim3(grid), dim3(256), 0, s, a);
  return hipGetLastError();
}

template <int EPI>
hipError_t launch_a8(const GemmArgs& a, hipStream_t s) {
  return a.w_group == KT ? launch_t<8, EPI, true>(a, s) : launch_t<8, EPI, false>(a, s);
}

}  // namespace

hipError_t launch_gemm(int act_bits, int epi, const GemmArgs& a, hipStream_t s) {
  if (act_bits == 8) {
    switch (epi) {
      case kEpiOut: return launch_a8<kEpiOut>(a, s);
      case kEpiPartial: return launch_a8<kEpiPartial>(a, s);
      case kEpiInt32: return launch_t<8, kEpiInt32, false>(a, s);
      case kEpiDump: return launch_a8<kEpiDump>(a, s);
    }
  } else {
    switch (epi) {
      case kEpiOut: return launch_t<4, kEpiOut, false>(a, s);
      case kEpiPartial: return launch_t<4, kEpiPartial, false>(a, s);
      case kEpiDump: return launch_t<4, kEpiDump, false>(a, s);
    }
  }
  return hipErrorInvalidValue;
}

}  // namespace sq
