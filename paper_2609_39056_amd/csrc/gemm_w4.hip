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
constexpr int A8_PITCH = KT + 16;     // LDS bytes per int8 activation row
constexpr int P_PITCH = KT / 2 + 8;   // LDS bytes per packed int4 row
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

template <int ABITS, int EPI>
__global__ __launch_bounds__(256) void gemm_w4_kernel(GemmArgs a) {
  constexpr int A_PITCH = ABITS == 8 ? A8_PITCH : P_PITCH;
  constexpr int A_ROW_BYTES = ABITS == 8 ? KT : KT / 2;     // per stage
  constexpr int A_CPR = A_ROW_BYTES / 16;                    // 16-byte chunks per row
  constexpr int A_PER_T = BM * A_CPR / 256;                  // chunks per thread
  constexpr int B_PER_T = BN * (KT / 2 / 16) / 256;          // 2
  constexpr bool NEED_SCALE = (EPI == kEpiOut || EPI == kEpiPartial);

  __shared__ __align__(16) uint8_t sA[2][BM * A_PITCH];
  __shared__ __align__(16) uint8_t sB[2][BN * P_PITCH];
  __shared__ __align__(16) float sS[2][ABITS == 4 ? 2 : 1][BM];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int M = a.M, N = a.N, K = a.K;

  const int ntm = (M + BM - 1) / BM;
  const int ntn = (N + BN - 1) / BN;
  int tile_m, tile_n;
  tile_of(ntm, ntn, tile_m, tile_n);
  const int m0 = tile_m * BM;
  const int n0 = tile_n * BN;
  const int nkt = K / KT;
  const size_t a_row_bytes = ABITS == 8 ? static_cast<size_t>(K) : static_cast<size_t>(K / 2);
  const size_t b_row_bytes = static_cast<size_t>(K / 2);
  const int nwg = K / a.w_group;  // weight groups per output channel

  const uint8_t* qx = static_cast<const uint8_t*>(a.qx);

  uint4 ra[A_PER_T];
  uint4 rb[B_PER_T];
  uint32_t rs = 0;  // two fp16 sigma of this thread's row (4-bit)

  auto load_stage = [&](int kt) {
#pragma unroll
    for (int p = 0; p < A_PER_T; ++p) {
      const int q = tid + p * 256;
      const int row = q / A_CPR, cc = q % A_CPR;
      const int grow = min(m0 + row, M - 1);
      ra[p] = *reinterpret_cast<const uint4*>(qx + grow * a_row_bytes + kt * A_ROW_BYTES + cc * 16);
    }
#pragma unroll
    for (int p = 0; p < B_PER_T; ++p) {
      const int q = tid + p * 256;
      const int col = q >> 2, cc = q & 3;
      const int gcol = min(n0 + col, N - 1);
      rb[p] = *reinterpret_cast<const uint4*>(a.qw + gcol * b_row_bytes + kt * (KT / 2) + cc * 16);
    }
    if constexpr (ABITS == 4 && NEED_SCALE) {
      if (tid < BM) {
        const int grow = min(m0 + tid, M - 1);
        const uint16_t* sp = static_cast<const uint16_t*>(a.act_scale) +
                             static_cast<size_t>(grow) * (K / kA4Group) + kt * 2;
        rs = *reinterpret_cast<const uint32_t*>(sp);
      }
    }
  };

  auto store_stage = [&](int buf) {
#pragma unroll
    for (int p = 0; p < A_PER_T; ++p) {
      const int q = tid + p * 256;
      const int row = q / A_CPR, cc = q % A_CPR;
      uint8_t* dst = &sA[buf][row * A_PITCH + cc * 16];
      if constexpr (ABITS == 8) {
        *reinterpret_cast<uint4*>(dst) = ra[p];
      } else {
        *reinterpret_cast<uint2*>(dst) = make_uint2(ra[p].x, ra[p].y);
        *reinterpret_cast<uint2*>(dst + 8) = make_uint2(ra[p].z, ra[p].w);
      }
    }
#pragma unroll
    for (int p = 0; p < B_PER_T; ++p) {
      const int q = tid + p * 256;
      const int col = q >> 2, cc = q & 3;
      uint8_t* dst = &sB[buf][col * P_PITCH + cc * 16];
      *reinterpret_cast<uint2*>(dst) = make_uint2(rb[p].x, rb[p].y);
      *reinterpret_cast<uint2*>(dst + 8) = make_uint2(rb[p].z, rb[p].w);
    }
    if constexpr (ABITS == 4 && NEED_SCALE) {
      if (tid < BM) {
        // sigma / 256 undoes the two factors of 16 of the widened codes (exact)
        sS[buf][0][tid] = f16_to_f32(rs & 0xFFFFu) * 0.00390625f;
        sS[buf][1][tid] = f16_to_f32(rs >> 16) * 0.00390625f;
      }
    }
  };

  // Output-channel columns owned by this lane, one per 32-wide tile.
  int gcol_t[TN];
#pragma unroll
  for (int tn = 0; tn < TN; ++tn) gcol_t[tn] = min(n0 + wn * 64 + tn * 32 + (lane & 31), N - 1);

  // Weight step of the current weight group for each owned column.  For
  // 8-bit activations the 1/16 of the widened weight codes is folded in.
  float wsv[TN];
  auto load_wscale = [&](int kt) {
    const int wb = (kt * KT) / a.w_group;
#pragma unroll
    for (int tn = 0; tn < TN; ++tn) {
      const float s = f16_to_f32(a.w_scale[static_cast<size_t>(gcol_t[tn]) * nwg + wb]);
      wsv[tn] = ABITS == 8 ? s * 0.0625f : s;
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

  // Write int32 block accumulators (test hook / unfused int32 path).
  auto dump_acc = [&](int blk) {
    int32_t* out = static_cast<int32_t*>(a.out);
    constexpr int SHIFT = ABITS == 8 ? 4 : 8;
#pragma unroll
    for (int tm = 0; tm < TM; ++tm)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int m = m0 + wm * 64 + tm * 32 + (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3);
        if (m >= M) continue;
#pragma unroll
        for (int tn = 0; tn < TN; ++tn) {
          const int n = n0 + wn * 64 + tn * 32 + (lane & 31);
          if (n < N) out[(static_cast<size_t>(blk) * M + m) * N + n] = acc[tm][tn][r] >> SHIFT;
        }
      }
  };

  load_stage(0);
  store_stage(0);
  __syncthreads();

  for (int kt = 0; kt < nkt; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nkt) load_stage(kt + 1);
    if constexpr (NEED_SCALE) load_wscale(kt);
    const bool fresh8 = ((kt * KT) % a.w_group) == 0;  // 8-bit: a new block starts here

    const uint8_t* A = sA[cur];
    const uint8_t* B = sB[cur];
#pragma unroll
    for (int ks = 0; ks < KT / 32; ++ks) {
      v4i af[TM], bf[TN];
#pragma unroll
      for (int tm = 0; tm < TM; ++tm) {
        const int row = wm * 64 + tm * 32 + (lane & 31);
        if constexpr (ABITS == 8) {
          af[tm] = *reinterpret_cast<const v4i*>(A + row * A_PITCH + ks * 32 + (lane >> 5) * 16);
        } else {
          af[tm] = unpack_frag(*reinterpret_cast<const uint2*>(A + row * A_PITCH + ks * 16 + (lane >> 5) * 8));
        }
      }
#pragma unroll
      for (int tn = 0; tn < TN; ++tn) {
        const int col = wn * 64 + tn * 32 + (lane & 31);
        bf[tn] = unpack_frag(*reinterpret_cast<const uint2*>(B + col * P_PITCH + ks * 16 + (lane >> 5) * 8));
      }
      const bool fresh = ABITS == 8 ? (ks == 0 && fresh8) : ((ks & 1) == 0);
#pragma unroll
      for (int tm = 0; tm < TM; ++tm)
#pragma unroll
        for (int tn = 0; tn < TN; ++tn) {
          if (fresh)
            acc[tm][tn] = __builtin_amdgcn_mfma_i32_32x32x32_i8(af[tm], bf[tn], (v16i)(0), 0, 0, 0);
          else
            acc[tm][tn] = __builtin_amdgcn_mfma_i32_32x32x32_i8(af[tm], bf[tn], acc[tm][tn], 0, 0, 0);
        }

      if constexpr (ABITS == 4) {
        if ((ks & 1) == 1) {  // end of a 64-wide block
          const int h = ks >> 1;
          if constexpr (EPI == kEpiDump) {
            dump_acc(kt * 2 + h);
          } else {
#pragma unroll
            for (int tm = 0; tm < TM; ++tm)
#pragma unroll
              for (int r4 = 0; r4 < 4; ++r4) {
                const int ml = wm * 64 + tm * 32 + r4 * 8 + (lane >> 5) * 4;
                const float4 sg = *reinterpret_cast<const float4*>(&sS[cur][h][ml]);
                const float sv[4] = {sg.x, sg.y, sg.z, sg.w};
#pragma unroll
                for (int tn = 0; tn < TN; ++tn)
#pragma unroll
                  for (int i = 0; i < 4; ++i) {
                    const int r = r4 * 4 + i;
                    const float t = static_cast<float>(acc[tm][tn][r]) * sv[i];
                    y[tm][tn][r] = __builtin_fmaf(t, wsv[tn], y[tm][tn][r]);
                  }
              }
          }
        }
      }
    }

    if constexpr (ABITS == 8) {
      if (((kt + 1) * KT) % a.w_group == 0) {  // end of a weight group
        if constexpr (EPI == kEpiDump) {
          dump_acc(((kt + 1) * KT) / a.w_group - 1);
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

    if (kt + 1 < nkt) store_stage(cur ^ 1);
    __syncthreads();
  }

  if constexpr (EPI == kEpiInt32) {
    dump_acc(0);
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

template <int ABITS, int EPI>
hipError_t launch_t(const GemmArgs& a, hipStream_t s) {
  const unsigned grid = static_cast<unsigned>(((a.M + BM - 1) / BM) * ((a.N + BN - 1) / BN));
  hipLaunchKernelGGL((gemm_w4_kernel<ABITS, EPI>), dim3(grid), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm(int act_bits, int epi, const GemmArgs& a, hipStream_t s) {
  if (act_bits == 8) {
    switch (epi) {
      case kEpiOut: return launch_t<8, kEpiOut>(a, s);
      case kEpiPartial: return launch_t<8, kEpiPartial>(a, s);
      case kEpiInt32: return launch_t<8, kEpiInt32>(a, s);
      case kEpiDump: return launch_t<8, kEpiDump>(a, s);
    }
  } else {
    switch (epi) {
      case kEpiOut: return launch_t<4, kEpiOut>(a, s);
      case kEpiPartial: return launch_t<4, kEpiPartial>(a, s);
      case kEpiDump: return launch_t<4, kEpiDump>(a, s);
    }
  }
  return hipErrorInvalidValue;
}

}  // namespace sq
