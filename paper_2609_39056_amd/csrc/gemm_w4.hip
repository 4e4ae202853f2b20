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
// Tiling.  A 256-thread workgroup (4 waves, 2 x 2) computes a 128 x 128 output
// tile; each wave owns 64 x 64 = 2 x 2 tiles of v_mfma_i32_32x32x32_i8.  K
// advances in stages of 128 channels.  Every byte a stage needs (activation
// codes, packed weights, group steps, weight steps) is copied straight from
// global memory into an LDS ring by global_load_lds (no registers, no LDS
// stores); the loads run two stages ahead and each stage ends with one
// explicit vmcnt wait and one barrier.  LDS rows are XOR-swizzled so that the
// 16-byte fragment reads are free of bank conflicts.
//
// Dequantization.  One int32 accumulator per K-block (the 128-wide weight
// group for 8-bit activations, 64 for 4-bit).  A block's MFMAs run tile by
// tile; just before a tile's first MFMA of block b + 1 its accumulator of
// block b is folded into the fp32 sum, so the VALU folding one tile overlaps
// the matrix cores working on the previous one: y += fp32(C) * Delta_W (8-bit;
// the row scale r_i factors out and is applied once in the epilogue; the
// block's int32 sum starts from a float bias, so that one full-rate
// subtraction converts it) or
// y += (fp32(C) * sigma_i) * Delta_W (4-bit).  The epilogue multiplies by r_i (8-bit) or by
// kappa_i = 1/gamma_s(i) (4-bit, the compensation of Eq. 8), adds the bias and
// casts.  With one weight step per output channel (w_group = K, the weight
// format of the paper's experiments) and 8-bit activations there is a single
// block: the int32 sums run over all of K and are converted once per tile.
#include <algorithm>
#include <atomic>
#include <cmath>
#include <type_traits>

#include "gemm_frag.h"
#include "gelu.h"
#include "sq_internal.h"

namespace sq {
namespace {

constexpr int TM = 2;        // 32-row MFMA tiles per wave
constexpr int TN = 2;        // 32-col MFMA tiles per wave
constexpr int GROUP_M = 8;   // m-tiles per supertile (L2 reuse)
constexpr bool kPipeWide = false;  // tile shape of the pipelined kernel (see Cfg)
constexpr bool kPipe16 = true;     // 8-bit, 128-wide groups: the GEMM on 16 x 16 x 64 MFMAs (gemm_pipe16_kernel)

// Workgroup shape: NWM x NWN waves of 64 x 64 outputs (the most a wave's
// registers hold: an int32 accumulator and an fp32 sum per output); a
// STAGES-deep LDS ring loaded DIST stages ahead.  The 4-bit path folds a block
// from the previous stage during the current one, which must therefore
// outlive the loads DIST stages ahead: one more stage.
//   WIDE: 128 x 256 tiles, 8 waves, one workgroup per CU, loads three stages
//   ahead.  A third fewer operand bytes per MFMA, but both waves on a SIMD
//   then belong to one workgroup and stall at its barriers together; measured
//   slower than two independent 128 x 128 workgroups per CU (kPipeWide).
//   otherwise: 128 x 128 tiles, 4 waves, two workgroups per CU, loads two
//   stages ahead.
template <int ABITS, bool WIDE = false>
struct Cfg {
  static constexpr int NWM = 2, NWN = WIDE ? 4 : 2;
  static constexpr int NWAVE = NWM * NWN;
  static constexpr int NTHREADS = NWAVE * 64;
  static constexpr int BM = 64 * NWM;
  static constexpr int BN = 64 * NWN;
  static constexpr int DIST = WIDE ? 3 : 2;
  static constexpr int STAGES = DIST + (ABITS == 8 ? 1 : 2);
  static constexpr int WGS_PER_CU = WIDE ? 1 : 2;
};

// Workgroup -> output tile.  Workgroups are dealt to the 8 XCDs round-robin;
// xcd_order renumbers the first n of them so that each XCD runs a contiguous
// range of logical tiles, and supertile walks the logical range in supertiles
// of GROUP_M m-tiles, so that tiles running at the same time on one XCD share
// activation rows and weight columns in its L2.
__device__ __forceinline__ int xcd_order(int bid, int n) {
  const int q = n / 8, r = n % 8;
  const int xcd = bid % 8, i = bid / 8;
  return xcd * q + min(xcd, r) + i;
}

__device__ __forceinline__ void supertile(int lid, int ntm, int ntn, int& tm, int& tn) {
  const int per_group = GROUP_M * ntn;
  const int group = lid / per_group;
  const int first_m = group * GROUP_M;
  const int gm = min(ntm - first_m, GROUP_M);
  const int in_group = lid % per_group;
  tm = first_m + in_group % gm;
  tn = in_group / gm;
}

// Work item `it` of a persistent pipelined GEMM: the output tiles computed
// whole (the first ndp of the logical order, XCD-ordered) followed by the K
// ranges of the split tail tiles.  Tile origin and K range [kt0, kt1); unit
// >= 0 numbers a split range.
struct PipeItem {
  int m0, n0, kt0, kt1, unit;
};
__device__ __forceinline__ PipeItem pipe_item(const GemmArgs& a, int it, int ntm, int ntn, int nkt, int BM, int BN) {
  PipeItem r;
  int lid;
  if (it < a.ndp) {
    lid = xcd_order(it, a.ndp);
    r.kt0 = 0;
    r.kt1 = nkt;
    r.unit = -1;
  } else {
    r.unit = it - a.ndp;
    lid = a.ndp + r.unit / a.split;
    const int sl = r.unit % a.split;
    r.kt0 = sl * nkt / a.split;
    r.kt1 = (sl + 1) * nkt / a.split;
  }
  int tm, tn;
  supertile(lid, ntm, ntn, tm, tn);
  r.m0 = tm * BM;
  r.n0 = tn * BN;
  return r;
}

// Wait until at most N of this wave's vector-memory operations are in flight
// and all of its LDS reads are done, then synchronize the workgroup: after it
// the stage about to be read has landed and no wave still reads the slot the
// next loads (or the epilogue) will overwrite.  One asm block with a memory
// clobber: no LDS access moves across it (a fenced __syncthreads would instead
// drain every outstanding load, including the stages still in flight).
template <int N>
__device__ __forceinline__ void wait_vm_and_barrier() {
  asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(N) : "memory");
}

// LDS layout of one pipeline stage (no padding; 16-byte chunks XOR-swizzled
// so that the fragment reads of 16 consecutive rows hit 16 distinct bank
// groups):
//   8-bit activations: row r (128 B) holds chunk c at position c ^ ((r >> 1) & 7)
//   packed int4 rows (weights, 4-bit activations; 64 B): c at c ^ ((r >> 2) & 3)
//   4-bit group steps: wave w loads rows R*w .. R*w+R-1 (R = BM / waves; the
//     64 lanes repeat them); the dword of row r (its two fp16 steps of this
//     stage) is at (r / R) * 256 + (r % R) * 4
//   weight steps (group-major in memory): wave w, lane i < 32 -> the dword
//     holding the fp16 steps of output channels wn * 64 + 2i, +1, at
//     w * 256 + i * 4 (lanes 32..63 load the same dwords again)
// Lane (row, h = lane >> 5) feeds MFMA k-step s (0..3) of a stage with the
// channels [64 (s >> 1) + 32 h + 16 (s & 1), +16): for 8-bit activations the
// 16-byte chunk 4 (s >> 1) + 2 h + (s & 1); for packed rows the low (s even)
// or high (s odd) half of chunk 2 (s >> 1) + h, so one 16-byte read serves two
// k-steps.  Activations and weights use the same assignment, so every product
// pairs equal channels, and k-steps {0, 1} cover channels [0, 64), {2, 3}
// cover [64, 128): a 64-wide block never straddles an MFMA.
template <int ABITS, bool WIDE>
struct Layout {
  using CF = Cfg<ABITS, WIDE>;
  static constexpr int A_BYTES = ABITS == 8 ? CF::BM * KT : CF::BM * KT / 2;
  static constexpr int B_BYTES = CF::BN * KT / 2;
  static constexpr int S_BYTES = ABITS == 4 ? CF::NWAVE * 256 : 0;
  static constexpr int W_BYTES = CF::NWAVE * 256;
  static constexpr int STAGE = A_BYTES + B_BYTES + S_BYTES + W_BYTES;
  static constexpr int A_DMA = A_BYTES / 1024 / CF::NWAVE;  // 16-byte loads per wave per stage
  static constexpr int B_DMA = B_BYTES / 1024 / CF::NWAVE;
  static constexpr int S_ROWS = CF::BM / CF::NWAVE;          // group-step rows loaded per wave
};

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

// Row factor of output row m0 + wm * 64 + lane (8-bit: r_i; 4-bit: the
// inverse gain kappa_i; 1 for partial sums) and the bias of the lane's two
// columns, loaded when a tile starts so that their latency hides under its
// main loop.  The GELU epilogue (8-bit) also loads the next layer's gain of
// that row, its 1 / Delta and the D^-1 of the four columns the lane holds
// after the quad transpose in each 32-wide tile.
template <int ABITS, int EPI>
struct EpiInputs {
  static constexpr bool kOut = EPI == kEpiOut || EPI == kEpiGelu;
  static constexpr bool kGelu = EPI == kEpiGelu;
  float rowf;
  float bias[TN];
  float gain, inv, delta;  // the next layer's gain of the row, 1 / Delta and (4-bit) Delta
  float dinv[kGelu ? TN : 1][4];
  __device__ __forceinline__ void load(const GemmArgs& a, int m0, int n0, int wm, int wn, int lane) {
    const int m = min(m0 + wm * 64 + lane, a.M - 1);
    rowf = 1.0f;
    if constexpr (kOut) {
      if constexpr (ABITS == 8) {
        rowf = static_cast<const float*>(a.act_scale)[m];
      } else {
        rowf = 1.0f / a.gamma[a.step * a.S + a.tok2stream[m]];
      }
    }
#pragma unroll
    for (int tn = 0; tn < TN; ++tn) {
      const int n = min(n0 + wn * 64 + tn * 32 + (lane & 31), a.N - 1);
      bias[tn] = (kOut && a.bias != nullptr) ? bf16_to_f32(a.bias[n]) : 0.0f;
    }
    if constexpr (kGelu) {
      const NextQuant& q = a.nq;
      gain = q.gamma[q.step * q.S + q.tok2stream[m]];
      if constexpr (ABITS == 8) {
        inv = 1.0f / (q.clip[q.step] / 127.0f);
        if (__builtin_isinf(inv)) inv = 0.0f;
      } else {
        static_step4(q.clip[q.step], delta, inv);
      }
#pragma unroll
      for (int tn = 0; tn < TN; ++tn) {
        const int n = min(n0 + wn * 64 + tn * 32 + (lane & 28), a.N - 4);
        const float4 d = q.dinv != nullptr ? *reinterpret_cast<const float4*>(q.dinv + n)
                                           : make_float4(1.0f, 1.0f, 1.0f, 1.0f);
        dinv[tn][0] = d.x;
        dinv[tn][1] = d.y;
        dinv[tn][2] = d.z;
        dinv[tn][3] = d.w;
      }
    }
  }
};

// Epilogue of one 128 x 128 output tile, from registers: row factor, bias,
// cast, store.  In the MFMA layout a lane holds one column and, for each group
// g of four registers, four consecutive rows; a quad transpose turns that into
// one row and four consecutive columns, so each lane writes 16 bytes (fp32) or
// 8 bytes (16-bit outputs) and eight lanes cover a row's 32 columns.  The row
// factors are fetched from the lane that loaded them (ds_bpermute).
template <int ABITS, int EPI>
__device__ __forceinline__ void store_tile(const GemmArgs& a, float (&y)[TM][TN][16], int m0, int n0, int wm,
                                           int wn, int lane_in, const EpiInputs<ABITS, EPI>& in) {
  // An opaque copy of the lane index: the per-lane values below are then
  // computed here, not hoisted out of a surrounding tile loop (where they
  // would hold registers through the whole main loop).
  int lane = lane_in;
  asm volatile("" : "+v"(lane));
  const int M = a.M, N = a.N;
  if (n0 + wn * 64 >= N) return;  // N % 64 == 0: a wave's 64 columns are all in or all out
  const bool f32out = EPI == kEpiPartial || a.out_dtype == SQ_OUT_F32;
  const int rf_bits = __float_as_int(in.rowf);
  const int half = (lane >> 5) * 16;  // lanes 32..63 hold rows 4 further down
  if constexpr (EPI == kEpiGelu && ABITS == 8) {  // the next layer's row scales, from the waves of the first column tile
    const int m = m0 + wm * 64 + lane;
    if (n0 + wn * 64 == 0 && m < M) a.nq.r[m] = (a.nq.clip[a.nq.step] / 127.0f) / in.gain;
  }
  if constexpr (EPI == kEpiGelu && ABITS == 4) {
    // the next layer's 4-bit codes as fp8 bytes, and per (row, 64-group) the
    // step sigma (fp32) and kc = -8 S sigma 2^-18 (S: the group's code sum);
    // the wave's 64 columns are one group, a row's codes sit in the lanes that
    // differ in bits 2-4 (both 32-wide tiles)
#pragma unroll
    for (int tm = 0; tm < TM; ++tm) {
      float rowf[16];
#pragma unroll
      for (int r = 0; r < 16; ++r)
        rowf[r] = __int_as_float(__builtin_amdgcn_ds_bpermute(half + (tm * 32 + (r >> 2) * 8 + (r & 3)) * 4, rf_bits));
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int m = m0 + wm * 64 + tm * 32 + g * 8 + (lane >> 5) * 4 + (lane & 3);
        const float gain = __int_as_float(__builtin_amdgcn_ds_bpermute(
            (tm * 32 + g * 8 + (lane >> 5) * 4 + (lane & 3)) * 4, __float_as_int(in.gain)));
        int csum = 0;
#pragma unroll
        for (int tn = 0; tn < TN; ++tn) {
          float v[4];
#pragma unroll
          for (int q = 0; q < 4; ++q) v[q] = __builtin_fmaf(y[tm][tn][g * 4 + q], rowf[g * 4 + q], in.bias[tn]);
          quad_transpose(v, lane);
          uint32_t bits[4], neg[4], w = 0;
          gelu_codes4_a4(v, in.dinv[tn], gain, in.inv, bits, neg);
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            int code;
            w |= fp8_code_byte(bits[j], neg[j], code) << (8 * j);
            csum += code;
          }
          const int n = n0 + wn * 64 + tn * 32 + (lane & 28);
          if (m < M) *reinterpret_cast<uint32_t*>(static_cast<uint8_t*>(a.out) + static_cast<size_t>(m) * N + n) = w;
        }
        csum += __shfl_xor(csum, 4, 64);
        csum += __shfl_xor(csum, 8, 64);
        csum += __shfl_xor(csum, 16, 64);
        if (m < M && (lane & 28) == 0) {
          const size_t gi = static_cast<size_t>(m) * (N / 64) + (n0 + wn * 64) / 64;
          static_cast<float*>(a.nq.scale)[gi] = in.delta;
          a.nq.kc[gi] = (static_cast<float>(-8 * csum) * in.delta) * 3.814697265625e-06f;  // * 2^-18
        }
      }
    }
    return;
  }
#pragma unroll
  for (int tm = 0; tm < TM; ++tm) {
    float rowf[16];
#pragma unroll
    for (int r = 0; r < 16; ++r)
      rowf[r] = __int_as_float(__builtin_amdgcn_ds_bpermute(half + (tm * 32 + (r >> 2) * 8 + (r & 3)) * 4, rf_bits));
#pragma unroll
    for (int tn = 0; tn < TN; ++tn)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        float v[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int r = g * 4 + q;
          v[q] = EPI == kEpiPartial ? y[tm][tn][r] : __builtin_fmaf(y[tm][tn][r], rowf[r], in.bias[tn]);
        }
        quad_transpose(v, lane);
        const int m = m0 + wm * 64 + tm * 32 + g * 8 + (lane >> 5) * 4 + (lane & 3);
        const int n = n0 + wn * 64 + tn * 32 + (lane & 28);
        float gain = 0.0f;  // the next layer's gain of the lane's row after the transpose
        if constexpr (EPI == kEpiGelu)
          gain = __int_as_float(__builtin_amdgcn_ds_bpermute(
              (tm * 32 + g * 8 + (lane >> 5) * 4 + (lane & 3)) * 4, __float_as_int(in.gain)));
        if (m < M) {
          if constexpr (EPI == kEpiGelu && ABITS == 8) {
            *reinterpret_cast<uint32_t*>(static_cast<int8_t*>(a.out) + static_cast<size_t>(m) * N + n) =
                gelu_codes4(v, in.dinv[tn], gain, in.inv);
          } else if (f32out) {
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
}

// A split range's sums of one BM x BN tile (unit `unit` of the partial
// buffer, row-major, rows past M not written), in the MFMA layout.
template <int BM, int BN>
__device__ __forceinline__ void write_partial(const GemmArgs& a, const float (&y)[TM][TN][16], int unit, int m0, int wm,
                                              int wn, int lane_in) {
  int ln = lane_in;  // opaque copy: keep the addresses out of the tile loop's live registers
  asm volatile("" : "+v"(ln));
  float* P = a.partial + static_cast<size_t>(unit) * BM * BN;
#pragma unroll
  for (int tm = 0; tm < TM; ++tm)
#pragma unroll
    for (int tn = 0; tn < TN; ++tn)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = wm * 64 + tm * 32 + (r >> 2) * 8 + (ln >> 5) * 4 + (r & 3);
        if (m0 + row < a.M) P[row * BN + wn * 64 + tn * 32 + (ln & 31)] = y[tm][tn][r];
      }
}

// Per-lane LDS read offsets of the MFMA fragments within a stage.  The swizzle
// terms depend on the lane only, since every wave's first row and column are
// multiples of 16, and a 32-row (32-column) step leaves them unchanged: the
// offsets of the second row (column) tile are the first's plus a constant,
// which the LDS reads take as an immediate.
template <int ABITS, bool WIDE>
struct FragOffsets {
  static constexpr int A_TILE_STEP = ABITS == 8 ? 32 * KT : 32 * (KT / 2);
  static constexpr int B_TILE_STEP = 32 * (KT / 2);
  int a0[4];
  int b0[2];
  __device__ __forceinline__ FragOffsets(int wm, int wn, int lane) {
    const int h = lane >> 5;
    const int arow0 = wm * 64 + (lane & 31);
    const int bcol0 = wn * 64 + (lane & 31);
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      if constexpr (ABITS == 8)
        a0[ks] = arow0 * KT + 16 * ((4 * (ks >> 1) + 2 * h + (ks & 1)) ^ ((arow0 >> 1) & 7));
      else
        a0[ks] = arow0 * (KT / 2) + 16 * ((2 * (ks >> 1) + h) ^ ((arow0 >> 2) & 3));
    }
#pragma unroll
    for (int k2 = 0; k2 < 2; ++k2)
      b0[k2] = Layout<ABITS, WIDE>::A_BYTES + bcol0 * (KT / 2) + 16 * ((2 * k2 + h) ^ ((bcol0 >> 2) & 3));
  }
  __device__ __forceinline__ int a(int tm, int ks) const { return a0[ks] + tm * A_TILE_STEP; }
  __device__ __forceinline__ int b(int tn, int k2) const { return b0[k2] + tn * B_TILE_STEP; }
};

// This wave's direct loads of one stage: per-lane 32-bit offsets within the
// tile (rows and columns past the matrix are clamped to the last one) and the
// wave's LDS destinations.
template <int ABITS, bool WIDE>
struct StageLoads {
  using LY = Layout<ABITS, WIDE>;
  uint32_t voffA[LY::A_DMA];
  uint32_t voffB[LY::B_DMA];
  uint32_t voffS;
  uint32_t wcol2;  // first of the two output channels whose fp16 steps this lane's dword holds

  __device__ __forceinline__ void set(int m0, int n0, int M, int N, int K, int wave, int wn, int lane) {
    const uint32_t a_row_bytes = ABITS == 8 ? K : K / 2;
#pragma unroll
    for (int i = 0; i < LY::A_DMA; ++i) {
      if constexpr (ABITS == 8) {
        const int row = 8 * (LY::A_DMA * wave + i) + (lane >> 3);
        const int c = (lane & 7) ^ ((row >> 1) & 7);
        voffA[i] = static_cast<uint32_t>(min(m0 + row, M - 1) - m0) * a_row_bytes + c * 16;
      } else {
        const int row = 16 * (LY::A_DMA * wave + i) + (lane >> 2);
        const int c = (lane & 3) ^ ((row >> 2) & 3);
        voffA[i] = static_cast<uint32_t>(min(m0 + row, M - 1) - m0) * a_row_bytes + c * 16;
      }
    }
#pragma unroll
    for (int i = 0; i < LY::B_DMA; ++i) {
      const int col = 16 * (LY::B_DMA * wave + i) + (lane >> 2);
      const int c = (lane & 3) ^ ((col >> 2) & 3);
      voffB[i] = static_cast<uint32_t>(min(n0 + col, N - 1) - n0) * static_cast<uint32_t>(K / 2) + c * 16;
    }
    voffS = 0;
    if constexpr (ABITS == 4) {
      const int row = LY::S_ROWS * wave + (lane % LY::S_ROWS);
      voffS = static_cast<uint32_t>(min(m0 + row, M - 1) - m0) * static_cast<uint32_t>((K / kA4Group) * 2);
    }
    // N is even, so the pair is clamped inside the row
    wcol2 = static_cast<uint32_t>(min(n0 + wn * 64 + 2 * (lane & 31), N - 2));
  }

  // stage kt of the tile at (m0, n0) into the ring slot at LDS address st
  template <bool SIGMA, bool STEPS>
  __device__ __forceinline__ void issue(const GemmArgs& a, int m0, int n0, int kt, uint32_t st, int wave) const {
    const int K = a.K;
    const uint8_t* bA = static_cast<const uint8_t*>(a.qx) +
                        static_cast<size_t>(m0) * (ABITS == 8 ? K : K / 2) + kt * (ABITS == 8 ? KT : KT / 2);
    const uint8_t* bB = a.qw + static_cast<size_t>(n0) * (K / 2) + kt * (KT / 2);
#pragma unroll
    for (int i = 0; i < LY::A_DMA; ++i) dma<16>(bA, voffA[i], st + (LY::A_DMA * wave + i) * 1024);
#pragma unroll
    for (int i = 0; i < LY::B_DMA; ++i) dma<16>(bB, voffB[i], st + LY::A_BYTES + (LY::B_DMA * wave + i) * 1024);
    if constexpr (SIGMA) {
      const uint8_t* bS = static_cast<const uint8_t*>(a.act_scale) + static_cast<size_t>(m0) * (K / kA4Group) * 2 + kt * 4;
      dma<4>(bS, voffS, st + LY::A_BYTES + LY::B_BYTES + wave * 256);
    }
    if constexpr (STEPS) {
      const uint32_t e = static_cast<uint32_t>((kt * KT) / a.w_group) * static_cast<uint32_t>(a.N) + wcol2;
      dma<4>(a.w_scale, e * 2, st + LY::A_BYTES + LY::B_BYTES + LY::S_BYTES + wave * 256);
    }
  }
};

// Weight steps of a stage for the wave's columns, widened-code factor folded in.
template <int ABITS, bool WIDE>
__device__ __forceinline__ void read_wscale(const uint8_t* st, int wave, int lane, float (&w)[TN]) {
  using LY = Layout<ABITS, WIDE>;
  constexpr float WFOLD = ABITS == 8 ? 0.0625f : 0.00390625f;  // 1/16 or 1/256
  const uint32_t* Wst = reinterpret_cast<const uint32_t*>(st + LY::A_BYTES + LY::B_BYTES + LY::S_BYTES + wave * 256);
#pragma unroll
  for (int tn = 0; tn < TN; ++tn) {
    const int c = tn * 32 + (lane & 31);  // column within the wave's 64
    const uint32_t pair = Wst[c >> 1];
    w[tn] = f16_to_f32((c & 1) ? (pair >> 16) : (pair & 0xFFFFu)) * WFOLD;
  }
}

// y += (fp32(C) * sigma_row) * Delta_W for row tile tm and both column tiles
// (4-bit activations); sigma of block half hb from the stage at st
template <int ABITS, bool WIDE>
__device__ __forceinline__ void fold4(float (&y)[TM][TN][16], const uint8_t* st, int hb, const v16i (&c)[TN], int wm,
                                      int tm, int lane, const float (&w)[TN]) {
  using LY = Layout<ABITS, WIDE>;
  const uint8_t* S = st + LY::A_BYTES + LY::B_BYTES;
#pragma unroll
  for (int r4 = 0; r4 < 4; ++r4) {
    const int ml = wm * 64 + tm * 32 + r4 * 8 + (lane >> 5) * 4;
    const uint4 sp = *reinterpret_cast<const uint4*>(S + (ml / LY::S_ROWS) * 256 + (ml % LY::S_ROWS) * 4);
    const uint32_t w4[4] = {sp.x, sp.y, sp.z, sp.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const uint32_t pair = w4[i];
#pragma unroll
      for (int tn = 0; tn < TN; ++tn) {
        const int r = r4 * 4 + i;
        const float cf = static_cast<float>(c[tn][r]);
        y[tm][tn][r] = __builtin_fmaf(hb ? mul_step16<1>(cf, pair) : mul_step16<0>(cf, pair), w[tn], y[tm][tn][r]);
      }
    }
  }
}

// The pipelined GEMM (8-bit activations with one weight step per 128 input
// channels, and 4-bit activations): persistent workgroups.  Work items are the
// output tiles computed whole (the first ndp of the logical order) followed by
// the K ranges of the split tail tiles; workgroup g takes items g, g + G,
// g + 2G, ...  The loads run two stages ahead along the workgroup's whole item
// sequence, so the next tile's first stages are in flight during the current
// tile's epilogue, and the epilogue's stores drain while the next tile
// computes.  Workgroups never wait for one another.
//
// 8-bit activations, one block per stage, tile-major: for each 32 x 32 tile,
// fold the previous block's accumulator into y, then run the tile's four MFMAs
// of this block; the fold of the next tile (VALU) overlaps these MFMAs.
// 4-bit activations: blocks are the two halves of a stage, row-tile-major:
// fold the previous block's accumulators of a row tile (they share its group
// steps), then run its MFMAs of this block; four stages, since the previous
// stage's group steps are still read while the stage two ahead loads.
template <int ABITS, int EPI, bool PC>
__global__ __launch_bounds__(kPipeWide ? 512 : 256, kPipeWide ? 1 : 2) void gemm_pipe_kernel(GemmArgs a) {
  using LY = Layout<ABITS, kPipeWide>;
  using CF = Cfg<ABITS, kPipeWide>;
  static_assert(CF::NTHREADS == (kPipeWide ? 512 : 256) && CF::WGS_PER_CU == (kPipeWide ? 1 : 2), "launch bounds");
  static_assert(!PC || ABITS == 8, "one weight step per channel: 8-bit activations (4-bit ones have 64-wide steps)");
  constexpr int BM = CF::BM, BN = CF::BN, STAGES = CF::STAGES;
  constexpr bool A4 = ABITS == 4;
  constexpr int NDMA = LY::A_DMA + LY::B_DMA + (A4 ? 1 : 0) + (PC ? 0 : 1);
  constexpr int AHEAD = (CF::DIST - 1) * NDMA;  // loads issued after the stage waited for
  constexpr uint32_t RING = STAGES * LY::STAGE;
  static_assert(EPI == kEpiOut || EPI == kEpiPartial || (EPI == kEpiGelu && ABITS == 8),
                "the pipelined path applies the weight steps");

  __shared__ __align__(1024) uint8_t smem[RING];

  const int lane = threadIdx.x & 63;
  // wave-uniform (an SGPR): keeps every per-wave LDS and global address scalar
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = wave / CF::NWN, wn = wave % CF::NWN;
  const int M = a.M, N = a.N, K = a.K;
  const int ntm = (M + BM - 1) / BM, ntn = (N + BN - 1) / BN, nkt = K / KT;
  const int nitems = a.ndp + (ntm * ntn - a.ndp) * a.split;
  const int G = gridDim.x;
  if (static_cast<int>(blockIdx.x) >= nitems) return;
  const uint32_t smem_lds = lds_offset(smem);
  if constexpr (A4) {
    // An item's first fold scales the previous slot's group steps by a zero
    // weight step; the steps there are another item's (finite) or, before
    // the ring's first use, these zeros: never a NaN or infinity.
    for (int i = threadIdx.x; i < STAGES * (LY::S_BYTES / 4); i += CF::NTHREADS) {
      const int s = i / (LY::S_BYTES / 4), e = i % (LY::S_BYTES / 4);
      reinterpret_cast<uint32_t*>(smem + s * LY::STAGE + LY::A_BYTES + LY::B_BYTES)[e] = 0u;
    }
    __syncthreads();
  }

  auto item_of = [&](int it) { return pipe_item(a, it, ntm, ntn, nkt, BM, BN); };

  // ---- the load cursor: (item, stage) two stages ahead of the computation
  int d_it = blockIdx.x;
  PipeItem d = item_of(d_it);
  int d_kt = d.kt0;
  uint32_t d_slot = 0;  // byte offset of the ring slot the next stage goes to
  StageLoads<ABITS, kPipeWide> ld;
  ld.set(d.m0, d.n0, M, N, K, wave, wn, lane);
  auto issue = [&]() {
    ld.template issue<A4, !PC>(a, d.m0, d.n0, d_kt, smem_lds + d_slot, wave);
    d_slot = d_slot + LY::STAGE == RING ? 0 : d_slot + LY::STAGE;
  };
  // Past the last stage of the last item the same stage is loaded again (in
  // bounds, into a free slot), so every iteration issues the same loads.
  auto advance = [&]() {
    if (d_kt + 1 < d.kt1) {
      ++d_kt;
    } else if (d_it + G < nitems) {
      d_it += G;
      d = item_of(d_it);
      d_kt = d.kt0;
      ld.set(d.m0, d.n0, M, N, K, wave, wn, lane);
    }
  };

  const FragOffsets<ABITS, kPipeWide> off(wm, wn, lane);

#pragma unroll
  for (int i = 0; i < CF::DIST; ++i) {
    issue();
    advance();
  }
  wait_vm_and_barrier<AHEAD>();

  uint32_t c_slot = 0;  // byte offset of the ring slot of the stage being computed
  auto next_slot = [&](uint32_t s) { return s + LY::STAGE == RING ? 0u : s + LY::STAGE; };
  auto prev_slot = [&](uint32_t s) { return s == 0 ? RING - LY::STAGE : s - LY::STAGE; };

  // The accumulators are set once: each tile's first fold scales whatever they
  // hold (finite integers) by a zero step.
  v16i acc[TM][TN];
#pragma unroll
  for (int tm = 0; tm < TM; ++tm)
#pragma unroll
    for (int tn = 0; tn < TN; ++tn) acc[tm][tn] = (v16i)(0);
  // 8-bit activations, 128-wide groups: each block's sum starts from the bits
  // of 1.5 * 2^23 (fold8_biased); |16 C| <= 128 * 128 * 128 = 2^21 for any
  // int8 codes, inside the exact range
  const v16i magic = (v16i)(kMagicAcc);
  for (int it = blockIdx.x;;) {
    const PipeItem c = item_of(it);
    EpiInputs<ABITS, EPI> ein;
    ein.load(a, c.m0, c.n0, wm, wn, lane);
    float y[TM][TN][16];
    float wsv_prev[TN], wsv[TN];
    if constexpr (!PC) {
#pragma unroll
      for (int tm = 0; tm < TM; ++tm)
#pragma unroll
        for (int tn = 0; tn < TN; ++tn)
#pragma unroll
          for (int r = 0; r < 16; ++r) y[tm][tn][r] = 0.0f;
#pragma unroll
      for (int tn = 0; tn < TN; ++tn) wsv_prev[tn] = 0.0f;  // the fold before the first block adds 0
    }

    if constexpr (PC) {
      // One weight step per output channel (w_group = K): the int32 sums of
      // the item's whole K range stay in the accumulators and are converted
      // once, after its last stage; the loop is MFMAs, the weight widening
      // and the loads only.  A split range hands its exact int32 sums to the
      // second kernel (as raw bits in y), which adds them in integers.
      float wpc[TN];
#pragma unroll
      for (int tn = 0; tn < TN; ++tn) {
        const int n = min(c.n0 + wn * 64 + tn * 32 + (lane & 31), N - 1);
        wpc[tn] = f16_to_f32(a.w_scale[n]) * 0.0625f;  // the widened codes' factor 16 folded in
      }
#pragma unroll
      for (int tm = 0; tm < TM; ++tm)
#pragma unroll
        for (int tn = 0; tn < TN; ++tn) acc[tm][tn] = (v16i)(0);
      for (int kt = c.kt0; kt < c.kt1; ++kt) {
        issue();
        advance();
        const uint8_t* st = smem + c_slot;
        v4i bfull[TN][4];
#pragma unroll
        for (int tn = 0; tn < TN; ++tn)
#pragma unroll
          for (int k2 = 0; k2 < 2; ++k2) {
            const uint4 pb = *reinterpret_cast<const uint4*>(st + off.b(tn, k2));
            bfull[tn][2 * k2] = unpack_frag(pb.x, pb.y);
            bfull[tn][2 * k2 + 1] = unpack_frag(pb.z, pb.w);
          }
        __builtin_amdgcn_s_setprio(1);  // the MFMA phase first at the arbiter (+2 %)
#pragma unroll
        for (int tm = 0; tm < TM; ++tm) {
          v4i af[4];
#pragma unroll
          for (int ks = 0; ks < 4; ++ks) af[ks] = *reinterpret_cast<const v4i*>(st + off.a(tm, ks));
#pragma unroll
          for (int tn = 0; tn < TN; ++tn)
#pragma unroll
            for (int ks = 0; ks < 4; ++ks)
              acc[tm][tn] = __builtin_amdgcn_mfma_i32_32x32x32_i8(af[ks], bfull[tn][ks], acc[tm][tn], 0, 0, 0);
        }
        __builtin_amdgcn_s_setprio(0);
        wait_vm_and_barrier<AHEAD>();
        c_slot = next_slot(c_slot);
      }
#pragma unroll
      for (int tm = 0; tm < TM; ++tm)
#pragma unroll
        for (int tn = 0; tn < TN; ++tn)
#pragma unroll
          for (int r = 0; r < 16; ++r)
            y[tm][tn][r] = c.unit >= 0 ? __int_as_float(acc[tm][tn][r]) : static_cast<float>(acc[tm][tn][r]) * wpc[tn];
    } else if constexpr (!A4) {
      for (int kt = c.kt0; kt < c.kt1; ++kt) {
        issue();
        advance();
        const uint8_t* st = smem + c_slot;
        read_wscale<ABITS, kPipeWide>(st, wave, lane, wsv);
        v4i bfull[TN][4];
#pragma unroll
        for (int tn = 0; tn < TN; ++tn)
#pragma unroll
          for (int k2 = 0; k2 < 2; ++k2) {
            const uint4 pb = *reinterpret_cast<const uint4*>(st + off.b(tn, k2));
            bfull[tn][2 * k2] = unpack_frag(pb.x, pb.y);
            bfull[tn][2 * k2 + 1] = unpack_frag(pb.z, pb.w);
          }
#pragma unroll
        for (int tm = 0; tm < TM; ++tm) {
          v4i af[4];
#pragma unroll
          for (int ks = 0; ks < 4; ++ks) af[ks] = *reinterpret_cast<const v4i*>(st + off.a(tm, ks));
#pragma unroll
          for (int tn = 0; tn < TN; ++tn) {
            fold8_biased(acc[tm][tn], wsv_prev[tn], y[tm][tn]);
            acc[tm][tn] = __builtin_amdgcn_mfma_i32_32x32x32_i8(af[0], bfull[tn][0], magic, 0, 0, 0);
#pragma unroll
            for (int ks = 1; ks < 4; ++ks)
              acc[tm][tn] = __builtin_amdgcn_mfma_i32_32x32x32_i8(af[ks], bfull[tn][ks], acc[tm][tn], 0, 0, 0);
          }
        }
        // issue order: each MFMA followed by a share of the VALU work (folds,
        // unpacking), so the VALU runs under the matrix cores
#pragma unroll
        for (int i = 0; i < TM * TN * 4; ++i) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // one MFMA
          __builtin_amdgcn_sched_group_barrier(0x002, 10, 0);  // up to ten VALU
        }
#pragma unroll
        for (int tn = 0; tn < TN; ++tn) wsv_prev[tn] = wsv[tn];
        wait_vm_and_barrier<AHEAD>();
        c_slot = next_slot(c_slot);
      }
#pragma unroll
      for (int t = 0; t < TM * TN; ++t) fold8_biased(acc[t / TN][t % TN], wsv_prev[t % TN], y[t / TN][t % TN]);
    } else {
      for (int kt = c.kt0; kt < c.kt1; ++kt) {
        issue();
        advance();
        const uint8_t* st = smem + c_slot;
        const uint8_t* st_prev = smem + prev_slot(c_slot);
        read_wscale<ABITS, kPipeWide>(st, wave, lane, wsv);
#pragma unroll
        for (int hb = 0; hb < 2; ++hb) {
          v4i bf[TN][2];
#pragma unroll
          for (int tn = 0; tn < TN; ++tn) {
            const uint4 pb = *reinterpret_cast<const uint4*>(st + off.b(tn, hb));
            bf[tn][0] = unpack_frag(pb.x, pb.y);
            bf[tn][1] = unpack_frag(pb.z, pb.w);
          }
#pragma unroll
          for (int tm = 0; tm < TM; ++tm) {
            const uint4 pa = *reinterpret_cast<const uint4*>(st + off.a(tm, 2 * hb));
            const v4i af0 = unpack_frag(pa.x, pa.y);
            const v4i af1 = unpack_frag(pa.z, pa.w);
            // previous block: second half of the previous stage, or first half of this one
            if (hb == 0) {
              fold4<ABITS, kPipeWide>(y, st_prev, 1, acc[tm], wm, tm, lane, wsv_prev);
            } else {
              fold4<ABITS, kPipeWide>(y, st, 0, acc[tm], wm, tm, lane, wsv);
            }
#pragma unroll
            for (int tn = 0; tn < TN; ++tn) {
              acc[tm][tn] = __builtin_amdgcn_mfma_i32_32x32x32_i8(af0, bf[tn][0], (v16i)(0), 0, 0, 0);
              acc[tm][tn] = __builtin_amdgcn_mfma_i32_32x32x32_i8(af1, bf[tn][1], acc[tm][tn], 0, 0, 0);
            }
          }
        }
#pragma unroll
        for (int tn = 0; tn < TN; ++tn) wsv_prev[tn] = wsv[tn];
        wait_vm_and_barrier<AHEAD>();
        c_slot = next_slot(c_slot);
      }
      const uint8_t* st_last = smem + prev_slot(c_slot);
#pragma unroll
      for (int tm = 0; tm < TM; ++tm) fold4<ABITS, kPipeWide>(y, st_last, 1, acc[tm], wm, tm, lane, wsv_prev);
    }

    if (c.unit >= 0) {
      // split tail: this K range's fp32 sums (int32 with one step per channel)
      write_partial<BM, BN>(a, y, c.unit, c.m0, wm, wn, lane);
    } else {
      store_tile<ABITS, EPI>(a, y, c.m0, c.n0, wm, wn, lane, ein);
    }
    it += G;
    if (it >= nitems) break;
  }
  // drain the loads still in flight (the re-issued last stages) before the
  // workgroup ends
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
}

// ---------------------------------------------------------------- 8-bit activations on 16 x 16 MFMA tiles
// The pipelined 8-bit GEMM with 128-wide weight groups on
// v_mfma_i32_16x16x64_i8: the same tiles, work list, loads, LDS layout, stage
// barrier and split tail as gemm_pipe_kernel, with each wave's 64 x 64
// outputs as 4 x 4 tiles of 16 x 16 (two MFMAs of 64 channels per 128-channel
// stage, each block's fold on four registers per tile).  In a register-only
// loop with random int8 operands and the per-block fold this instruction
// sustains about 1.5x the rate of the 32 x 32 x 32 one under the board's power
// limit; in the GEMM it gains 0-5 % (2B up about equal, 2B and 14B down 2-5 %
// faster).  With one weight step per channel (PC: no fold, int32 sums over
// all of K, converted once with the column's step) it was as fast as the
// 32 x 32 kernel before the raised-priority MFMA phase and is 2 % faster with
// it on the 14B block (equal on the 2B layers); the 32 x 32 kernel stays for
// the fp32 partial sums of the unfused path, whose 16 x 16 stores cover half
// a line.
//
// Lane (row or column lane & 15, g = lane >> 4) feeds k-step s (0, 1) of a
// stage with the channels [32 g + 16 s, +16): for 8-bit activations the
// 16-byte chunk 2 g + s of the row, for packed weights the low (s = 0) or high
// (s = 1) half of chunk g of the column, so one 16-byte read serves both
// k-steps.  Both operands use the same assignment.  An accumulator lane holds
// column lane & 15 and rows 4 (lane >> 4) + j, j < 4.
//
// Waves: P16_NWM across a tile's 128 rows and P16_NWN across its 128
// columns, each computing P16_WROWS x P16_WCOLS outputs as TM16 x TN16 tiles
// of 16 x 16.  Measured alternatives to 2 x 2 waves of 64 x 64: 2 x 4 waves of
// 64 x 32 (four waves per SIMD) the same speed without the raised-priority
// MFMA phase below and 1 % slower with it, 1 x 4 waves of 128 x 32 (each
// weight fragment widened once per workgroup) 1-2 % slower.
constexpr int P16_NWM = 2, P16_NWN = 2;
constexpr int TM16 = 8 / P16_NWM, TN16 = 8 / P16_NWN;
constexpr int P16_WROWS = 16 * TM16, P16_WCOLS = 16 * TN16;
constexpr int P16_RH = P16_WROWS / 64;  // 64-row halves of a wave's rows (one row per lane each)
struct P16 {
  static constexpr int NWM = P16_NWM, NWN = P16_NWN, NWAVE = NWM * NWN, NTHREADS = NWAVE * 64;
  static constexpr int BM = 128, BN = 128;
  static constexpr int DIST = 2, STAGES = 3, WGS_PER_CU = 2;
  // one stage in LDS: A codes, packed weights, then each wave's 256-byte
  // area of weight-step pairs (the Layout<8, false> arrangement, except that
  // weight column n holds chunk c at position c ^ ((n >> 1) & 3): the 16
  // columns of a fragment read then fill all 64 banks; with (n >> 2) & 3 the
  // read took twice as long in an LDS probe, and the kernel gained 0.5 %)
  static constexpr int A_BYTES = BM * KT, B_BYTES = BN * KT / 2, W_BYTES = NWAVE * 256;
  static constexpr int STAGE = A_BYTES + B_BYTES + W_BYTES;
  static constexpr int A_DMA = A_BYTES / 1024 / NWAVE, B_DMA = B_BYTES / 1024 / NWAVE;
};
static_assert(P16::BM == Cfg<8, kPipeWide>::BM && P16::BN == Cfg<8, kPipeWide>::BN,
              "the split tail and the plan use the pipelined kernels' tile");

// This wave's direct loads of one stage (StageLoads' arrangement for P16's
// wave count; weight steps of 128-wide groups: stage kt is group kt).
struct StageLoads16 {
  uint32_t voffA[P16::A_DMA];
  uint32_t voffB[P16::B_DMA];
  uint32_t wcol2;  // first of the two output channels whose fp16 steps this lane's dword holds

  __device__ __forceinline__ void set(int m0, int n0, int M, int N, int K, int wave, int wn, int lane) {
#pragma unroll
    for (int i = 0; i < P16::A_DMA; ++i) {
      const int row = 8 * (P16::A_DMA * wave + i) + (lane >> 3);
      const int c = (lane & 7) ^ ((row >> 1) & 7);
      voffA[i] = static_cast<uint32_t>(min(m0 + row, M - 1) - m0) * static_cast<uint32_t>(K) + c * 16;
    }
#pragma unroll
    for (int i = 0; i < P16::B_DMA; ++i) {
      const int col = 16 * (P16::B_DMA * wave + i) + (lane >> 2);
      const int c = (lane & 3) ^ ((col >> 1) & 3);
      voffB[i] = static_cast<uint32_t>(min(n0 + col, N - 1) - n0) * static_cast<uint32_t>(K / 2) + c * 16;
    }
    // N is even, so the pair is clamped inside the row
    wcol2 = static_cast<uint32_t>(min(n0 + wn * P16_WCOLS + 2 * (lane & (P16_WCOLS / 2 - 1)), N - 2));
  }

  template <bool PC = false>
  __device__ __forceinline__ void issue(const GemmArgs& a, int m0, int n0, int kt, uint32_t st, int wave) const {
    const int K = a.K;
    const uint8_t* bA = static_cast<const uint8_t*>(a.qx) + static_cast<size_t>(m0) * K + kt * KT;
    const uint8_t* bB = a.qw + static_cast<size_t>(n0) * (K / 2) + kt * (KT / 2);
#pragma unroll
    for (int i = 0; i < P16::A_DMA; ++i) dma<16>(bA, voffA[i], st + (P16::A_DMA * wave + i) * 1024);
#pragma unroll
    for (int i = 0; i < P16::B_DMA; ++i) dma<16>(bB, voffB[i], st + P16::A_BYTES + (P16::B_DMA * wave + i) * 1024);
    if constexpr (!PC) {  // one step per channel: read once, in the epilogue
      const uint32_t e = static_cast<uint32_t>(kt) * static_cast<uint32_t>(a.N) + wcol2;
      dma<4>(a.w_scale, e * 2, st + P16::A_BYTES + P16::B_BYTES + wave * 256);
    }
  }
};

struct FragOffsets16 {
  int a0[2];
  int b0;
  __device__ __forceinline__ FragOffsets16(int wm, int wn, int lane) {
    using LY = P16;
    const int g = lane >> 4;
    const int arow0 = wm * P16_WROWS + (lane & 15);
    const int bcol0 = wn * P16_WCOLS + (lane & 15);
#pragma unroll
    for (int s = 0; s < 2; ++s) a0[s] = arow0 * KT + 16 * ((2 * g + s) ^ ((arow0 >> 1) & 7));
    b0 = LY::A_BYTES + bcol0 * (KT / 2) + 16 * (g ^ ((bcol0 >> 1) & 3));
  }
  // a 16-row step keeps the swizzle term ((row >> 1) & 7 and (col >> 1) & 3)
  __device__ __forceinline__ int a(int tm, int s) const { return a0[s] + tm * 16 * KT; }
  __device__ __forceinline__ int b(int tn) const { return b0 + tn * 16 * (KT / 2); }
};

// the weight steps of a stage for the lane's column of each 16-wide tile
__device__ __forceinline__ void read_wscale16(const uint8_t* st, int wave, int lane, float (&w)[TN16]) {
  const uint32_t* Wst = reinterpret_cast<const uint32_t*>(st + P16::A_BYTES + P16::B_BYTES + wave * 256);
#pragma unroll
  for (int tn = 0; tn < TN16; ++tn) {
    const int c = tn * 16 + (lane & 15);  // column within the wave's P16_WCOLS
    const uint32_t pair = Wst[c >> 1];
    w[tn] = f16_to_f32((c & 1) ? (pair >> 16) : (pair & 0xFFFFu)) * 0.0625f;  // widened codes: factor 16
  }
}

// Row factors of rows m0 + wm * P16_WROWS + 64 h + lane and the bias of the
// lane's column in each 16-wide tile, loaded when a tile starts.  The GELU epilogue also loads
// the next layer's gain of that row, its 1 / Delta and the D^-1 of the four
// columns the lane holds after the quad transpose in each 16-wide tile.
template <int EPI>
struct EpiInputs16 {
  static constexpr bool kOut = EPI == kEpiOut || EPI == kEpiGelu;
  static constexpr bool kGelu = EPI == kEpiGelu;
  float rowf[P16_RH];
  float bias[TN16];
  float gain[P16_RH];
  float inv;
  float dinv[kGelu ? TN16 : 1][4];
  __device__ __forceinline__ void load(const GemmArgs& a, int m0, int n0, int wm, int wn, int lane) {
#pragma unroll
    for (int h = 0; h < P16_RH; ++h) {
      const int m = min(m0 + wm * P16_WROWS + h * 64 + lane, a.M - 1);
      rowf[h] = kOut ? static_cast<const float*>(a.act_scale)[m] : 1.0f;
      if constexpr (kGelu) gain[h] = a.nq.gamma[a.nq.step * a.nq.S + a.nq.tok2stream[m]];
    }
#pragma unroll
    for (int tn = 0; tn < TN16; ++tn) {
      const int n = min(n0 + wn * P16_WCOLS + tn * 16 + (lane & 15), a.N - 1);
      bias[tn] = (kOut && a.bias != nullptr) ? bf16_to_f32(a.bias[n]) : 0.0f;
    }
    if constexpr (kGelu) {
      const NextQuant& q = a.nq;
      inv = 1.0f / (q.clip[q.step] / 127.0f);
      if (__builtin_isinf(inv)) inv = 0.0f;
#pragma unroll
      for (int tn = 0; tn < TN16; ++tn) {
        const int n = min(n0 + wn * P16_WCOLS + tn * 16 + (lane & 12), a.N - 4);
        const float4 d = q.dinv != nullptr ? *reinterpret_cast<const float4*>(q.dinv + n)
                                           : make_float4(1.0f, 1.0f, 1.0f, 1.0f);
        dinv[tn][0] = d.x;
        dinv[tn][1] = d.y;
        dinv[tn][2] = d.z;
        dinv[tn][3] = d.w;
      }
    }
  }
};

// Epilogue of one 128 x 128 tile from the 16 x 16 accumulator layout: row
// factor and bias per lane (one column, four rows), a quad transpose to one
// row and four consecutive columns, then 16-byte (fp32) or 8-byte stores; or,
// for the GELU epilogue, four code bytes of the next layer (4-byte stores)
// and, from the waves of the first column tile, the next layer's row scales.
template <int EPI>
__device__ __forceinline__ void store_tile16(const GemmArgs& a, float (&y)[TM16][TN16][4], int m0, int n0, int wm,
                                             int wn, int lane_in, const EpiInputs16<EPI>& in) {
  int lane = lane_in;
  asm volatile("" : "+v"(lane));
  const int M = a.M, N = a.N;
  // N % 64 == 0 and the waves' column ranges are 64-aligned or nest in 64:
  // a wave's columns are all in or all out
  if (n0 + wn * P16_WCOLS >= N) return;
  const bool f32out = EPI == kEpiPartial || a.out_dtype == SQ_OUT_F32;
  const int q4 = (lane >> 4) * 4;
  if constexpr (EPI == kEpiGelu) {
#pragma unroll
    for (int h = 0; h < P16_RH; ++h) {
      const int m = m0 + wm * P16_WROWS + h * 64 + lane;
      if (n0 + wn * P16_WCOLS == 0 && m < M) a.nq.r[m] = (a.nq.clip[a.nq.step] / 127.0f) / in.gain[h];
    }
  }
#pragma unroll
  for (int tm = 0; tm < TM16; ++tm) {
    const int h = tm / 4, t4 = tm % 4;  // the 64-row half and the 16-row tile within it
    const int rf_bits = __float_as_int(in.rowf[h]);
    float rowf[4];
#pragma unroll
    for (int j = 0; j < 4; ++j)
      rowf[j] = __int_as_float(__builtin_amdgcn_ds_bpermute((t4 * 16 + q4 + j) * 4, rf_bits));
    float gain = 0.0f;
    if constexpr (EPI == kEpiGelu)
      gain = __int_as_float(__builtin_amdgcn_ds_bpermute((t4 * 16 + q4 + (lane & 3)) * 4, __float_as_int(in.gain[h])));
#pragma unroll
    for (int tn = 0; tn < TN16; ++tn) {
      float v[4];
#pragma unroll
      for (int j = 0; j < 4; ++j)
        v[j] = EPI == kEpiPartial ? y[tm][tn][j] : __builtin_fmaf(y[tm][tn][j], rowf[j], in.bias[tn]);
      quad_transpose(v, lane);
      const int m = m0 + wm * P16_WROWS + tm * 16 + q4 + (lane & 3);
      const int n = n0 + wn * P16_WCOLS + tn * 16 + (lane & 12);
      if (m < M) {
        if constexpr (EPI == kEpiGelu) {
          *reinterpret_cast<uint32_t*>(static_cast<int8_t*>(a.out) + static_cast<size_t>(m) * N + n) =
              gelu_codes4(v, in.dinv[tn], gain, in.inv);
        } else if (f32out) {
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
}

// A split range's sums of one 128 x 128 tile in the layout of
// gemm_tail_kernel's partial buffer (row-major tile, rows past M not written).
__device__ __forceinline__ void write_partial16(const GemmArgs& a, const float (&y)[TM16][TN16][4], int unit, int m0,
                                                int wm, int wn, int lane_in) {
  constexpr int BM = P16::BM, BN = P16::BN;
  int ln = lane_in;
  asm volatile("" : "+v"(ln));
  float* P = a.partial + static_cast<size_t>(unit) * BM * BN;
#pragma unroll
  for (int tm = 0; tm < TM16; ++tm)
#pragma unroll
    for (int tn = 0; tn < TN16; ++tn)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int row = wm * P16_WROWS + tm * 16 + (ln >> 4) * 4 + j;
        if (m0 + row < a.M) P[row * BN + wn * P16_WCOLS + tn * 16 + (ln & 15)] = y[tm][tn][j];
      }
}

template <int EPI, bool PC>
__global__ __launch_bounds__(P16::NTHREADS, P16::WGS_PER_CU) void gemm_pipe16_kernel(GemmArgs a) {
  using LY = P16;
  using CF = P16;
  static_assert(EPI == kEpiOut || EPI == kEpiPartial || EPI == kEpiGelu,
                "the pipelined path applies the weight steps");
  constexpr int BM = CF::BM, BN = CF::BN;
  constexpr int NDMA = LY::A_DMA + LY::B_DMA + (PC ? 0 : 1);
  constexpr int AHEAD = (CF::DIST - 1) * NDMA;
  constexpr uint32_t RING = CF::STAGES * LY::STAGE;

  __shared__ __align__(1024) uint8_t smem[RING];

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = wave / CF::NWN, wn = wave % CF::NWN;
  const int M = a.M, N = a.N, K = a.K;
  const int ntm = (M + BM - 1) / BM, ntn = (N + BN - 1) / BN, nkt = K / KT;
  const int nitems = a.ndp + (ntm * ntn - a.ndp) * a.split;
  const int G = gridDim.x;
  if (static_cast<int>(blockIdx.x) >= nitems) return;
  const uint32_t smem_lds = lds_offset(smem);

  auto item_of = [&](int it) { return pipe_item(a, it, ntm, ntn, nkt, BM, BN); };

  // the load cursor: (item, stage) two stages ahead of the computation
  int d_it = blockIdx.x;
  PipeItem d = item_of(d_it);
  int d_kt = d.kt0;
  uint32_t d_slot = 0;
  StageLoads16 ld;
  ld.set(d.m0, d.n0, M, N, K, wave, wn, lane);
  auto issue = [&]() {
    ld.template issue<PC>(a, d.m0, d.n0, d_kt, smem_lds + d_slot, wave);
    d_slot = d_slot + LY::STAGE == RING ? 0 : d_slot + LY::STAGE;
  };
  // past the last stage of the last item the same stage is loaded again (in
  // bounds, into a free slot), so every iteration issues the same loads
  auto advance = [&]() {
    if (d_kt + 1 < d.kt1) {
      ++d_kt;
    } else if (d_it + G < nitems) {
      d_it += G;
      d = item_of(d_it);
      d_kt = d.kt0;
      ld.set(d.m0, d.n0, M, N, K, wave, wn, lane);
    }
  };

  const FragOffsets16 off(wm, wn, lane);
#pragma unroll
  for (int i = 0; i < CF::DIST; ++i) {
    issue();
    advance();
  }
  wait_vm_and_barrier<AHEAD>();

  uint32_t c_slot = 0;
  auto next_slot = [&](uint32_t s) { return s + LY::STAGE == RING ? 0u : s + LY::STAGE; };

  // the accumulators are set once: each tile's first fold scales whatever
  // they hold (finite values) by a zero step
  v4i acc[TM16][TN16];
#pragma unroll
  for (int tm = 0; tm < TM16; ++tm)
#pragma unroll
    for (int tn = 0; tn < TN16; ++tn) acc[tm][tn] = (v4i)(0);
  // each block's sum starts from the bits of 1.5 * 2^23 (fold8_biased4); |16 C|
  // <= 128 * 128 * 128 = 2^21 for any int8 codes, inside the exact range
  const v4i magic = (v4i)(kMagicAcc);
  for (int it = blockIdx.x;;) {
    const PipeItem c = item_of(it);
    EpiInputs16<EPI> ein;
    ein.load(a, c.m0, c.n0, wm, wn, lane);
    float y[TM16][TN16][4];
    if constexpr (PC) {
      // int32 sums over all of K (|16 C| < 2^31 for K <= 2^17), converted once
#pragma unroll
      for (int tm = 0; tm < TM16; ++tm)
#pragma unroll
        for (int tn = 0; tn < TN16; ++tn) acc[tm][tn] = (v4i)(0);
      for (int kt = c.kt0; kt < c.kt1; ++kt) {
        issue();
        advance();
        const uint8_t* st = smem + c_slot;
        v4i bq[TN16][2];
#pragma unroll
        for (int tn = 0; tn < TN16; ++tn) {
          const uint4 pb = *reinterpret_cast<const uint4*>(st + off.b(tn));
          bq[tn][0] = unpack_frag(pb.x, pb.y);
          bq[tn][1] = unpack_frag(pb.z, pb.w);
        }
        __builtin_amdgcn_s_setprio(1);
#pragma unroll
        for (int tm = 0; tm < TM16; ++tm) {
          const v4i a0 = *reinterpret_cast<const v4i*>(st + off.a(tm, 0));
          const v4i a1 = *reinterpret_cast<const v4i*>(st + off.a(tm, 1));
#pragma unroll
          for (int tn = 0; tn < TN16; ++tn) {
            acc[tm][tn] = __builtin_amdgcn_mfma_i32_16x16x64_i8(a0, bq[tn][0], acc[tm][tn], 0, 0, 0);
            acc[tm][tn] = __builtin_amdgcn_mfma_i32_16x16x64_i8(a1, bq[tn][1], acc[tm][tn], 0, 0, 0);
          }
        }
        __builtin_amdgcn_s_setprio(0);
        wait_vm_and_barrier<AHEAD>();
        c_slot = next_slot(c_slot);
      }
#pragma unroll
      for (int tn = 0; tn < TN16; ++tn) {
        const int n = min(c.n0 + wn * P16_WCOLS + tn * 16 + (lane & 15), N - 1);
        const float wpc = f16_to_f32(a.w_scale[n]) * 0.0625f;  // widened codes: factor 16
#pragma unroll
        for (int tm = 0; tm < TM16; ++tm)
#pragma unroll
          for (int j = 0; j < 4; ++j)
            y[tm][tn][j] = c.unit >= 0 ? __int_as_float(acc[tm][tn][j]) : static_cast<float>(acc[tm][tn][j]) * wpc;
      }
    } else {
      float wsv_prev[TN16], wsv[TN16];
#pragma unroll
      for (int tm = 0; tm < TM16; ++tm)
#pragma unroll
        for (int tn = 0; tn < TN16; ++tn)
#pragma unroll
          for (int j = 0; j < 4; ++j) y[tm][tn][j] = 0.0f;
#pragma unroll
      for (int tn = 0; tn < TN16; ++tn) wsv_prev[tn] = 0.0f;  // the fold before the first block adds 0
      for (int kt = c.kt0; kt < c.kt1; ++kt) {
        issue();
        advance();
        const uint8_t* st = smem + c_slot;
        read_wscale16(st, wave, lane, wsv);
        v4i bq[TN16][2];
#pragma unroll
        for (int tn = 0; tn < TN16; ++tn) {
          const uint4 pb = *reinterpret_cast<const uint4*>(st + off.b(tn));
          bq[tn][0] = unpack_frag(pb.x, pb.y);
          bq[tn][1] = unpack_frag(pb.z, pb.w);
        }
        // the MFMA phase at a raised wave priority: when both waves of a SIMD
        // can issue, the one feeding the matrix cores goes first and the
        // other's widening and folds fill the gaps (measured +8 % on the 14B
        // block against equal priorities)
        __builtin_amdgcn_s_setprio(1);
#pragma unroll
        for (int tm = 0; tm < TM16; ++tm) {
          const v4i a0 = *reinterpret_cast<const v4i*>(st + off.a(tm, 0));
          const v4i a1 = *reinterpret_cast<const v4i*>(st + off.a(tm, 1));
#pragma unroll
          for (int tn = 0; tn < TN16; ++tn) {
            fold8_biased4(acc[tm][tn], wsv_prev[tn], y[tm][tn]);
            acc[tm][tn] = __builtin_amdgcn_mfma_i32_16x16x64_i8(a0, bq[tn][0], magic, 0, 0, 0);
            acc[tm][tn] = __builtin_amdgcn_mfma_i32_16x16x64_i8(a1, bq[tn][1], acc[tm][tn], 0, 0, 0);
          }
        }
        // issue order: each tile's two MFMAs followed by a share of the VALU
        // work (folds), so the VALU runs under the matrix cores (with the raised
        // priority, pairs of MFMAs and ten VALU measured 2 % faster than single
        // MFMAs and five)
#pragma unroll
        for (int i = 0; i < TM16 * TN16; ++i) {
          __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);   // two MFMAs
          __builtin_amdgcn_sched_group_barrier(0x002, 10, 0);  // up to ten VALU
        }
        __builtin_amdgcn_s_setprio(0);
#pragma unroll
        for (int tn = 0; tn < TN16; ++tn) wsv_prev[tn] = wsv[tn];
        wait_vm_and_barrier<AHEAD>();
        c_slot = next_slot(c_slot);
      }
#pragma unroll
      for (int t = 0; t < TM16 * TN16; ++t)
        fold8_biased4(acc[t / TN16][t % TN16], wsv_prev[t % TN16], y[t / TN16][t % TN16]);
    }

    if (c.unit >= 0) {
      write_partial16(a, y, c.unit, c.m0, wm, wn, lane);
    } else {
      store_tile16<EPI>(a, y, c.m0, c.n0, wm, wn, lane, ein);
    }
    it += G;
    if (it >= nitems) break;
  }
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
}

// ---------------------------------------------------------------- 4-bit activations on the fp8 matrix cores
// The fused linear's 4-bit path for the tiled kernel.  The first kernel wrote
// each activation code as the fp8 e4m3 byte of code * 2^-9 (sign and
// magnitude; |code| <= 7 is an exact subnormal).  A packed weight nibble n
// (two's complement) XOR 8 is code + 8 in 0..15, and the fp8 byte with that
// value is (code + 8) * 2^-9 (subnormal below 8, normal above, one straight
// line).  v_mfma_f32_32x32x64_f8f6f4 multiplies and sums one 64-wide block
// exactly in fp32 (integers below 2^24 times 2^-18), giving
// C' = (C + 8 S) 2^-18 with S the block's activation code sum; the first
// kernel stored kc = -8 S sigma 2^-18 and sigma (fp32) per (row, block), so
// one fma(C', sigma, kc) is round(C sigma) 2^-18, the same value as the int8
// path's fp32(C) * sigma, and y += that * (Delta_W 2^18).  Per output and
// block: two full-rate fmas instead of a conversion, a v_fma_mix_f32 (half
// rate) and an fma, and no activation widening.
struct F8Layout {
  static constexpr int BM = 128, BN = 128, NWAVE = 4;
  static constexpr int A_BYTES = BM * KT;      // fp8 code rows of 128 B, chunk c at c ^ ((r >> 1) & 7)
  static constexpr int B_BYTES = BN * KT / 2;  // packed weight rows of 64 B, chunk c at c ^ ((r >> 2) & 3)
  static constexpr int B_OFF = A_BYTES;
  // fp32 group steps sigma and kc: row 32 w + i, block half b at w * 256 + b * 128 + i * 4
  static constexpr int SG_OFF = B_OFF + B_BYTES;
  static constexpr int KC_OFF = SG_OFF + NWAVE * 256;
  static constexpr int W_OFF = KC_OFF + NWAVE * 256;   // weight-step pairs: columns 2 i, 2 i + 1 at i * 4
  static constexpr int STAGE = W_OFF + 256;
  // loads run one stage ahead; the previous stage's steps are still read
  // while the current one is computed
  static constexpr int STAGES = 3;
  static constexpr int A_DMA = A_BYTES / 1024 / NWAVE, B_DMA = B_BYTES / 1024 / NWAVE;
};

struct F8Loads {
  using LY = F8Layout;
  uint32_t voffA[LY::A_DMA];
  uint32_t voffB[LY::B_DMA];
  uint32_t voffS, voffW;

  __device__ __forceinline__ void set(const GemmArgs& a, int m0, int n0, int wave, int lane) {
    const int M = a.M, N = a.N, K = a.K;
#pragma unroll
    for (int i = 0; i < LY::A_DMA; ++i) {
      const int row = 8 * (LY::A_DMA * wave + i) + (lane >> 3);
      const int c = (lane & 7) ^ ((row >> 1) & 7);
      voffA[i] = static_cast<uint32_t>(min(m0 + row, M - 1) - m0) * static_cast<uint32_t>(K) + c * 16;
    }
#pragma unroll
    for (int i = 0; i < LY::B_DMA; ++i) {
      const int col = 16 * (LY::B_DMA * wave + i) + (lane >> 2);
      const int c = (lane & 3) ^ ((col >> 2) & 3);
      voffB[i] = static_cast<uint32_t>(min(n0 + col, N - 1) - n0) * static_cast<uint32_t>(K / 2) + c * 16;
    }
    const uint32_t groups = static_cast<uint32_t>(K / kA4Group);
    // sigma and kc: lane -> row 32 wave + (lane & 31), block half lane >> 5
    voffS = static_cast<uint32_t>(min(m0 + 32 * wave + (lane & 31), M - 1) - m0) * groups * 4 + (lane >> 5) * 4;
    voffW = static_cast<uint32_t>(min(n0 + 2 * lane, N - 2));  // N is even: the pair stays in the row
  }

  // stage kt of the tile at (m0, n0) into the ring slot at LDS address st
  __device__ __forceinline__ void issue(const GemmArgs& a, int m0, int n0, int kt, uint32_t st, int wave) const {
    const int K = a.K;
    const size_t groups = static_cast<size_t>(K / kA4Group);
    const uint8_t* bA = static_cast<const uint8_t*>(a.qx) + static_cast<size_t>(m0) * K + kt * KT;
    const uint8_t* bB = a.qw + static_cast<size_t>(n0) * (K / 2) + kt * (KT / 2);
#pragma unroll
    for (int i = 0; i < LY::A_DMA; ++i) dma<16>(bA, voffA[i], st + (LY::A_DMA * wave + i) * 1024);
#pragma unroll
    for (int i = 0; i < LY::B_DMA; ++i) dma<16>(bB, voffB[i], st + LY::B_OFF + (LY::B_DMA * wave + i) * 1024);
    const uint8_t* bS = static_cast<const uint8_t*>(a.act_scale) + static_cast<size_t>(m0) * groups * 4 + kt * 8;
    dma<4>(bS, voffS, st + LY::SG_OFF + wave * 256);
    const uint8_t* bK = reinterpret_cast<const uint8_t*>(a.kc) + static_cast<size_t>(m0) * groups * 4 + kt * 8;
    dma<4>(bK, voffS, st + LY::KC_OFF + wave * 256);
    if (wave == 0) {
      const uint32_t e = static_cast<uint32_t>((kt * KT) / a.w_group) * static_cast<uint32_t>(a.N) + voffW;
      dma<4>(a.w_scale, e * 2, st + LY::W_OFF);
    }
  }
};

// fp8 operand of 32 weight codes: one packed 16-byte chunk -> code + 8 per byte
__device__ __forceinline__ v8i unpack_offset_frag(const uint4& p) {
  const uint32_t w[4] = {p.x, p.y, p.z, p.w};
  v8i r;
#pragma unroll
  for (int d = 0; d < 4; ++d) {
    // each nibble XOR 8 = code + 8 (mod 16); (x & m) ^ c is one three-input op
    r[2 * d] = static_cast<int>((w[d] & 0x0F0F0F0Fu) ^ 0x08080808u);
    r[2 * d + 1] = static_cast<int>(((w[d] >> 4) & 0x0F0F0F0Fu) ^ 0x08080808u);
  }
  return r;
}

// y += round(C sigma) * Delta_W for row tile tm and both column tiles, block
// half hb of the stage at st (w: Delta_W * 2^18 of the lane's two columns).
// The lane's rows are 64 wm + 32 tm + 8 r4 + 4 h + i: wave block 2 wm + tm,
// row 8 r4 + 4 h + i within it; `rowb` = wm * 512 + h * 16 (4 bytes of sigma
// or kc per row and block), the rest are immediate offsets.
__device__ __forceinline__ void fold_f8(float (&y)[TM][TN][16], const uint8_t* st, int hb, const v16f (&c)[TN],
                                        int rowb, int tm, const float (&w)[TN]) {
  using LY = F8Layout;
#pragma unroll
  for (int r4 = 0; r4 < 4; ++r4) {
    const int o = rowb + tm * 256 + r4 * 32;
    const uint4 sp = *reinterpret_cast<const uint4*>(st + LY::SG_OFF + o + hb * 128);
    const uint4 kq = *reinterpret_cast<const uint4*>(st + LY::KC_OFF + o + hb * 128);
    const uint32_t s4[4] = {sp.x, sp.y, sp.z, sp.w};
    const uint32_t kb[4] = {kq.x, kq.y, kq.z, kq.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float sg = __uint_as_float(s4[i]);
#pragma unroll
      for (int tn = 0; tn < TN; ++tn) {
        const int r = r4 * 4 + i;
        const float t = __builtin_fmaf(c[tn][r], sg, __uint_as_float(kb[i]));
        y[tm][tn][r] = __builtin_fmaf(t, w[tn], y[tm][tn][r]);
      }
    }
  }
}

template <int EPI>
__global__ __launch_bounds__(256, 2) void gemm_a4f8_kernel(GemmArgs a) {
  using LY = F8Layout;
  constexpr int BM = LY::BM, BN = LY::BN;
  constexpr uint32_t RING = LY::STAGES * LY::STAGE;
  static_assert(EPI == kEpiOut || EPI == kEpiPartial || EPI == kEpiGelu, "the pipelined path applies the weight steps");
  static_assert(2 * RING <= 160 * 1024, "two workgroups per CU");

  __shared__ __align__(1024) uint8_t smem[RING];

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = wave / 2, wn = wave % 2;
  const int M = a.M, N = a.N, K = a.K;
  const int ntm = (M + BM - 1) / BM, ntn = (N + BN - 1) / BN, nkt = K / KT;
  const int nitems = a.ndp + (ntm * ntn - a.ndp) * a.split;
  const int G = gridDim.x;
  if (static_cast<int>(blockIdx.x) >= nitems) return;
  const uint32_t smem_lds = lds_offset(smem);
  // An item's first fold scales the previous slot's steps by a zero weight
  // step: those are another item's (finite) or, before the ring's first use,
  // these zeros.
  for (int i = threadIdx.x; i < LY::STAGES * (2 * LY::NWAVE * 256 / 4); i += 256) {
    const int s = i / (2 * LY::NWAVE * 256 / 4), e = i % (2 * LY::NWAVE * 256 / 4);
    reinterpret_cast<uint32_t*>(smem + s * LY::STAGE + LY::SG_OFF)[e] = 0u;
  }
  __syncthreads();

  int d_it = blockIdx.x;
  PipeItem d = pipe_item(a, d_it, ntm, ntn, nkt, BM, BN);
  int d_kt = d.kt0;
  uint32_t d_slot = 0;
  F8Loads ld;
  ld.set(a, d.m0, d.n0, wave, lane);
  auto issue = [&]() {
    ld.issue(a, d.m0, d.n0, d_kt, smem_lds + d_slot, wave);
    d_slot = d_slot + LY::STAGE == RING ? 0 : d_slot + LY::STAGE;
  };
  // past the last stage of the last item the same stage is loaded again
  auto advance = [&]() {
    if (d_kt + 1 < d.kt1) {
      ++d_kt;
    } else if (d_it + G < nitems) {
      d_it += G;
      d = pipe_item(a, d_it, ntm, ntn, nkt, BM, BN);
      d_kt = d.kt0;
      ld.set(a, d.m0, d.n0, wave, lane);
    }
  };
  issue();
  advance();
  wait_vm_and_barrier<0>();

  // per-lane LDS offsets of the fragments (row tile 1 / column tile 1: + 32 rows)
  const int arow = wm * 64 + (lane & 31), bcol = wn * 64 + (lane & 31), h = lane >> 5;
  int aoff[2][2], boff[2];
#pragma unroll
  for (int hb = 0; hb < 2; ++hb) {
#pragma unroll
    for (int q = 0; q < 2; ++q) aoff[hb][q] = arow * KT + 16 * ((4 * hb + 2 * h + q) ^ ((arow >> 1) & 7));
    boff[hb] = LY::B_OFF + bcol * (KT / 2) + 16 * ((2 * hb + h) ^ ((bcol >> 2) & 3));
  }
  const int wc = wn * 64 + (lane & 31);  // the lane's first column within the tile
  int rowb = wm * 512 + h * 16;           // step / kc offset of the lane's first row (see fold_f8)
  asm volatile("" : "+v"(rowb));          // a per-lane base: keep the tile offsets as immediates

  uint32_t c_slot = 0;
  auto next_slot = [&](uint32_t s) { return s + LY::STAGE == RING ? 0u : s + LY::STAGE; };
  auto prev_slot = [&](uint32_t s) { return s == 0 ? RING - LY::STAGE : s - LY::STAGE; };
  auto read_w = [&](const uint8_t* st, float (&w)[TN]) {
    const uint32_t* W = reinterpret_cast<const uint32_t*>(st + LY::W_OFF);
#pragma unroll
    for (int tn = 0; tn < TN; ++tn) {
      const int col = wc + tn * 32;
      const uint32_t pair = W[col >> 1];
      w[tn] = f16_to_f32((col & 1) ? (pair >> 16) : (pair & 0xFFFFu)) * 262144.0f;  // * 2^18
    }
  };

  v16f acc[TM][TN];
#pragma unroll
  for (int tm = 0; tm < TM; ++tm)
#pragma unroll
    for (int tn = 0; tn < TN; ++tn) acc[tm][tn] = (v16f)(0.0f);
  for (int it = blockIdx.x;;) {
    const PipeItem c = pipe_item(a, it, ntm, ntn, nkt, BM, BN);
    EpiInputs<4, EPI> ein;
    ein.load(a, c.m0, c.n0, wm, wn, lane);
    float y[TM][TN][16];
#pragma unroll
    for (int tm = 0; tm < TM; ++tm)
#pragma unroll
      for (int tn = 0; tn < TN; ++tn)
#pragma unroll
        for (int r = 0; r < 16; ++r) y[tm][tn][r] = 0.0f;
    float wsv_prev[TN] = {0.0f, 0.0f}, wsv[TN];
    for (int kt = c.kt0; kt < c.kt1; ++kt) {
      issue();
      advance();
      const uint8_t* st = smem + c_slot;
      const uint8_t* st_prev = smem + prev_slot(c_slot);
      read_w(st, wsv);
#pragma unroll
      for (int hb = 0; hb < 2; ++hb) {
        v8i bf[TN];
#pragma unroll
        for (int tn = 0; tn < TN; ++tn)
          bf[tn] = unpack_offset_frag(*reinterpret_cast<const uint4*>(st + boff[hb] + tn * 32 * (KT / 2)));
        __builtin_amdgcn_s_setprio(1);  // the MFMA phase first at the arbiter (+1 %)
#pragma unroll
        for (int tm = 0; tm < TM; ++tm) {
          const uint4 a0 = *reinterpret_cast<const uint4*>(st + aoff[hb][0] + tm * 32 * KT);
          const uint4 a1 = *reinterpret_cast<const uint4*>(st + aoff[hb][1] + tm * 32 * KT);
          const v8i af = {static_cast<int>(a0.x), static_cast<int>(a0.y), static_cast<int>(a0.z),
                          static_cast<int>(a0.w), static_cast<int>(a1.x), static_cast<int>(a1.y),
                          static_cast<int>(a1.z), static_cast<int>(a1.w)};
          // previous block: second half of the previous stage, or first half of this one
          if (hb == 0) {
            fold_f8(y, st_prev, 1, acc[tm], rowb, tm, wsv_prev);
          } else {
            fold_f8(y, st, 0, acc[tm], rowb, tm, wsv);
          }
#pragma unroll
          for (int tn = 0; tn < TN; ++tn)
            acc[tm][tn] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(af, bf[tn], (v16f)(0.0f), 0, 0, 0, 0, 0, 0);
        }
      }
      __builtin_amdgcn_s_setprio(0);
#pragma unroll
      for (int tn = 0; tn < TN; ++tn) wsv_prev[tn] = wsv[tn];
      wait_vm_and_barrier<0>();
      c_slot = next_slot(c_slot);
    }
    const uint8_t* st_last = smem + prev_slot(c_slot);
#pragma unroll
    for (int tm = 0; tm < TM; ++tm) fold_f8(y, st_last, 1, acc[tm], rowb, tm, wsv_prev);

    if (c.unit >= 0) {
      write_partial<BM, BN>(a, y, c.unit, c.m0, wm, wn, lane);  // split tail: this K range's fp32 sums
    } else {
      store_tile<4, EPI>(a, y, c.m0, c.n0, wm, wn, lane, ein);
    }
    it += G;
    if (it >= nitems) break;
  }
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
}

// The non-pipelined GEMM: one output tile per workgroup, all of K.  Blocks are
// folded (or written out) when they end.  Used for 8-bit activations whose
// weight blocks span several stages (w_group > 128), and for the int32
// outputs (the unfused path's C and the test hook's block dump).
template <int ABITS, int EPI>
__global__ __launch_bounds__(Cfg<ABITS>::NTHREADS, 2) void gemm_simple_kernel(GemmArgs a) {
  using LY = Layout<ABITS, false>;
  using CF = Cfg<ABITS, false>;
  static_assert(CF::DIST == 2, "the loop below loads two stages ahead");
  constexpr int BM = CF::BM, BN = CF::BN, STAGES = CF::STAGES;
  constexpr bool NEED_SCALE = (EPI == kEpiOut || EPI == kEpiPartial);
  static_assert(!(NEED_SCALE && ABITS == 4), "4-bit activations with weight steps take the pipelined kernel");
  constexpr int NDMA = LY::A_DMA + LY::B_DMA + (NEED_SCALE ? 1 : 0);

  __shared__ __align__(1024) uint8_t smem[STAGES * LY::STAGE];

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = wave / CF::NWN, wn = wave % CF::NWN;
  const int M = a.M, N = a.N, K = a.K;
  const int ntm = (M + BM - 1) / BM, ntn = (N + BN - 1) / BN, nkt = K / KT;
  int tile_m, tile_n;
  supertile(xcd_order(blockIdx.x, gridDim.x), ntm, ntn, tile_m, tile_n);
  const int m0 = tile_m * BM;
  const int n0 = tile_n * BN;
  const uint32_t smem_lds = lds_offset(smem);

  StageLoads<ABITS, false> ld;
  ld.set(m0, n0, M, N, K, wave, wn, lane);
  // stage kt into slot kt % STAGES; past the last stage the source is clamped
  // to it (the slot written is free and never read again)
  auto issue_stage = [&](int kt_slot) {
    ld.template issue<false, NEED_SCALE>(a, m0, n0, min(kt_slot, nkt - 1), smem_lds + (kt_slot % STAGES) * LY::STAGE,
                                         wave);
  };
  const FragOffsets<ABITS, false> off(wm, wn, lane);

  float y[TM][TN][16];
  v16i acc[TM][TN];
#pragma unroll
  for (int tm = 0; tm < TM; ++tm)
#pragma unroll
    for (int tn = 0; tn < TN; ++tn) {
      acc[tm][tn] = (v16i)(0);
#pragma unroll
      for (int r = 0; r < 16; ++r) y[tm][tn][r] = 0.0f;
    }

  issue_stage(0);
  issue_stage(1);
  wait_vm_and_barrier<NDMA>();
  for (int kt = 0; kt < nkt; ++kt) {
    issue_stage(kt + 2);
    const uint8_t* st = smem + (kt % STAGES) * LY::STAGE;
    float wsv[TN];
    if constexpr (NEED_SCALE) read_wscale<ABITS, false>(st, wave, lane, wsv);
    if constexpr (ABITS == 8) {
      if ((kt * KT) % a.w_group == 0) {
#pragma unroll
        for (int tm = 0; tm < TM; ++tm)
#pragma unroll
          for (int tn = 0; tn < TN; ++tn) acc[tm][tn] = (v16i)(0);
      }
    }
    uint4 pa[TM], pb[TN];
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      v4i af[TM], bf[TN];
#pragma unroll
      for (int tm = 0; tm < TM; ++tm) {
        if constexpr (ABITS == 8) {
          af[tm] = *reinterpret_cast<const v4i*>(st + off.a(tm, ks));
        } else {
          if ((ks & 1) == 0) pa[tm] = *reinterpret_cast<const uint4*>(st + off.a(tm, ks));
          af[tm] = (ks & 1) ? unpack_frag(pa[tm].z, pa[tm].w) : unpack_frag(pa[tm].x, pa[tm].y);
        }
      }
#pragma unroll
      for (int tn = 0; tn < TN; ++tn) {
        if ((ks & 1) == 0) pb[tn] = *reinterpret_cast<const uint4*>(st + off.b(tn, ks >> 1));
        bf[tn] = (ks & 1) ? unpack_frag(pb[tn].z, pb[tn].w) : unpack_frag(pb[tn].x, pb[tn].y);
      }
      const bool zero_c = ABITS == 4 && (ks & 1) == 0;
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
        if ((ks & 1) == 1) dump_block<ABITS>(a, acc, kt * 2 + (ks >> 1), m0, n0, wm, wn, lane);
      }
    }
    if constexpr (ABITS == 8) {
      if (((kt + 1) * KT) % a.w_group == 0) {  // end of a weight group
        if constexpr (EPI == kEpiDump) {
          dump_block<ABITS>(a, acc, ((kt + 1) * KT) / a.w_group - 1, m0, n0, wm, wn, lane);
        } else if constexpr (NEED_SCALE) {
#pragma unroll
          for (int t = 0; t < TM * TN; ++t) fold8(acc[t / TN][t % TN], wsv[t % TN], y[t / TN][t % TN]);
        }
      }
    }
    wait_vm_and_barrier<NDMA>();
  }
  if constexpr (EPI == kEpiInt32) dump_block<ABITS>(a, acc, 0, m0, n0, wm, wn, lane);

  // drain the clamped loads issued by the last iterations before the LDS is
  // reused (or the workgroup ends)
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  if constexpr (NEED_SCALE) {
    EpiInputs<ABITS, EPI> ein;
    ein.load(a, m0, n0, wm, wn, lane);
    store_tile<ABITS, EPI>(a, y, m0, n0, wm, wn, lane, ein);
  }
}

// Second kernel of a split tail: adds the `split` partial sums of every
// output of the split tiles in range order (so the result does not depend on
// which range finished first) and finishes it exactly as store_tile does
// (one fma with the row factor and the bias, then the cast).  With one weight
// step per channel (PC) the partials are int32 sums, added exactly and then
// converted and scaled as the unsplit tile is.  Four adjacent outputs per
// thread, 16-byte loads.
template <int ABITS, int EPI, bool PC>
__global__ __launch_bounds__(256) void gemm_tail_kernel(GemmArgs a) {
  constexpr int BM = Cfg<ABITS, kPipeWide>::BM, BN = Cfg<ABITS, kPipeWide>::BN;
  constexpr int PER_TILE = BM * BN / 4;  // threads per tile
  const int g = blockIdx.x * 256 + threadIdx.x;
  const int ti = g / PER_TILE;
  const int e = (g % PER_TILE) * 4;
  const int row = e / BN, col = e % BN;
  const int ntm = (a.M + BM - 1) / BM;
  const int ntn = (a.N + BN - 1) / BN;
  int tile_m, tile_n;
  supertile(a.ndp + ti, ntm, ntn, tile_m, tile_n);
  const int m = tile_m * BM + row;
  const int n = tile_n * BN + col;
  if (m >= a.M || n >= a.N) return;  // N % 64 == 0: the 4 columns are all in or all out
  const float* P = a.partial + static_cast<size_t>(ti) * a.split * BM * BN + row * BN + col;
  // the epilogue's inputs first, so that their loads overlap the partial sums'
  constexpr bool kOut = EPI == kEpiOut || EPI == kEpiGelu;
  float rowf = 1.0f, bias[4] = {0.0f, 0.0f, 0.0f, 0.0f}, wpc[4];
  if constexpr (kOut) {
    rowf = ABITS == 8 ? static_cast<const float*>(a.act_scale)[m] : 1.0f / a.gamma[a.step * a.S + a.tok2stream[m]];
    if (a.bias != nullptr) {
#pragma unroll
      for (int j = 0; j < 4; ++j) bias[j] = bf16_to_f32(a.bias[n + j]);
    }
  }
  if constexpr (PC) {
#pragma unroll
    for (int j = 0; j < 4; ++j) wpc[j] = f16_to_f32(a.w_scale[n + j]) * 0.0625f;
  }
  const float4 acc = sum_ranges4<PC>(P, static_cast<size_t>(BM) * BN, a.split);
  float y[4] = {acc.x, acc.y, acc.z, acc.w};
  if constexpr (PC) {  // the int32 sums, converted once with the column's step
#pragma unroll
    for (int j = 0; j < 4; ++j) y[j] = static_cast<float>(__float_as_int(y[j])) * wpc[j];
  }
  if constexpr (kOut) {
#pragma unroll
    for (int j = 0; j < 4; ++j) y[j] = __builtin_fmaf(y[j], rowf, bias[j]);
  }
  if constexpr (EPI == kEpiGelu && ABITS == 4) {
    // fp8 code bytes; the 16 threads of a row's 64-group (lanes that differ in
    // bits 0-3) add their code sums, and the first writes sigma and kc
    const NextQuant& q = a.nq;
    const float gain = q.gamma[q.step * q.S + q.tok2stream[m]];
    float delta, inv;
    static_step4(q.clip[q.step], delta, inv);
    float d[4] = {1.0f, 1.0f, 1.0f, 1.0f};
    if (q.dinv != nullptr) {
      const float4 dv = *reinterpret_cast<const float4*>(q.dinv + n);
      d[0] = dv.x;
      d[1] = dv.y;
      d[2] = dv.z;
      d[3] = dv.w;
    }
    uint32_t bits[4], neg[4], w = 0;
    gelu_codes4_a4(y, d, gain, inv, bits, neg);
    int csum = 0;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      int code;
      w |= fp8_code_byte(bits[j], neg[j], code) << (8 * j);
      csum += code;
    }
    *reinterpret_cast<uint32_t*>(static_cast<uint8_t*>(a.out) + static_cast<size_t>(m) * a.N + n) = w;
    csum += __shfl_xor(csum, 1, 64);
    csum += __shfl_xor(csum, 2, 64);
    csum += __shfl_xor(csum, 4, 64);
    csum += __shfl_xor(csum, 8, 64);
    if ((n & 63) == 0) {
      const size_t gi = static_cast<size_t>(m) * (a.N / 64) + n / 64;
      static_cast<float*>(q.scale)[gi] = delta;
      q.kc[gi] = (static_cast<float>(-8 * csum) * delta) * 3.814697265625e-06f;  // * 2^-18
    }
    return;
  }
  if constexpr (EPI == kEpiGelu) {
    const NextQuant& q = a.nq;
    const float gain = q.gamma[q.step * q.S + q.tok2stream[m]];
    const float delta = q.clip[q.step] / 127.0f;
    float inv = 1.0f / delta;
    if (__builtin_isinf(inv)) inv = 0.0f;
    float d[4] = {1.0f, 1.0f, 1.0f, 1.0f};
    if (q.dinv != nullptr) {
      const float4 dv = *reinterpret_cast<const float4*>(q.dinv + n);
      d[0] = dv.x;
      d[1] = dv.y;
      d[2] = dv.z;
      d[3] = dv.w;
    }
    *reinterpret_cast<uint32_t*>(static_cast<int8_t*>(a.out) + static_cast<size_t>(m) * a.N + n) =
        gelu_codes4(y, d, gain, inv);
    if (n == 0) q.r[m] = delta / gain;
    return;
  }
  if (EPI == kEpiPartial || a.out_dtype == SQ_OUT_F32) {
    *reinterpret_cast<float4*>(static_cast<float*>(a.out) + static_cast<size_t>(m) * a.N + n) =
        make_float4(y[0], y[1], y[2], y[3]);
  } else {
    uint32_t h[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) h[j] = a.out_dtype == SQ_OUT_BF16 ? f32_to_bf16(y[j]) : f32_to_f16(y[j]);
    *reinterpret_cast<uint2*>(static_cast<uint16_t*>(a.out) + static_cast<size_t>(m) * a.N + n) =
        make_uint2(h[0] | (h[1] << 16), h[2] | (h[3] << 16));
  }
}

// Split plan of the pipelined kernel (tiles of BM x BN, `slots` workgroups at
// once): the tiles that fill whole rounds run whole; the R left over (all of
// them when there are fewer tiles than slots) are each split into S K ranges
// when that is faster.  In units of one stage of one tile on one workgroup,
// the split tail takes about nkt / S stages plus the partial sums' traffic,
// c * R * S with c = (rows * BN * 8 bytes written and read back) / (about
// 4.4 MB moved per stage time), plus about two for the extra launch;
// S ~ sqrt(nkt / (c R)), with ranges of >= 2 stages, R * S <= slots and R * S
// units of BM * BN floats fitting in `partial_bytes`.  Only the pipelined
// paths split (their blocks never straddle a range boundary).
struct Plan {
  int ntiles, ndp, split;
};
template <int BM, int BN>
Plan plan_split(bool pipe, int32_t M, int32_t N, int32_t K, int slots, size_t partial_bytes) {
  const int ntm = (M + BM - 1) / BM, ntn = (N + BN - 1) / BN;
  const int ntiles = ntm * ntn;
  Plan p{ntiles, ntiles, 1};
  const int nkt = K / KT;
  const int rest = ntiles % slots;
  if (!pipe || rest == 0 || nkt < 4) return p;
  // rows of a left-over tile: the left-over tiles are the last ones of the
  // logical order, which lie in the last row of tiles when there are few
  const int rows = (ntm == 1 || rest <= ntn) ? M - BM * (ntm - 1) : BM;
  const double c = rows * static_cast<double>(BN) * 8.0 / 4.4e6;
  int split = static_cast<int>(std::lround(std::sqrt(nkt / (c * rest))));
  split = std::min(std::min(split, nkt / 2), slots / rest);
  constexpr size_t unit = static_cast<size_t>(BM) * BN * sizeof(float);
  while (split >= 2 && static_cast<size_t>(rest) * split * unit > partial_bytes) --split;
  if (split < 2) return p;
  const double t_split = static_cast<double>(nkt) / split + c * rest * split + 2.0;
  if (t_split >= nkt) return p;
  p.ndp = ntiles - rest;
  p.split = split;
  return p;
}

template <int ABITS>
Plan pipe_plan(int32_t M, int32_t N, int32_t K, size_t partial_bytes) {
  using CF = Cfg<ABITS, kPipeWide>;
  return plan_split<CF::BM, CF::BN>(true, M, N, K, device_cus() * CF::WGS_PER_CU, partial_bytes);
}

template <int ABITS, int EPI, bool PIPE, bool PC = false>
hipError_t launch_t(const GemmArgs& a0, hipStream_t s, float* partial, size_t partial_bytes) {
  GemmArgs a = a0;
  if constexpr (PIPE) {
    using CF = Cfg<ABITS, kPipeWide>;
    const int slots = device_cus() * CF::WGS_PER_CU;
    const Plan p = pipe_plan<ABITS>(a.M, a.N, a.K, partial ? partial_bytes : 0);
    a.ndp = p.ndp;
    a.split = p.split;
    a.partial = p.split > 1 ? partial : nullptr;
    const int rest = p.ntiles - p.ndp;
    const int nitems = p.ndp + rest * p.split;
    const unsigned grid = static_cast<unsigned>(std::min(nitems, slots));
    if constexpr (ABITS == 8 && (EPI == kEpiOut || EPI == kEpiGelu) && kPipe16) {
      hipLaunchKernelGGL((gemm_pipe16_kernel<EPI, PC>), dim3(grid), dim3(P16::NTHREADS), 0, s, a);
    } else
      hipLaunchKernelGGL((gemm_pipe_kernel<ABITS, EPI, PC>), dim3(grid), dim3(CF::NTHREADS), 0, s, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || rest == 0 || p.split == 1) return e;
    constexpr int per_tile_blocks = CF::BM * CF::BN / 4 / 256;
    hipLaunchKernelGGL((gemm_tail_kernel<ABITS, EPI, PC>), dim3(rest * per_tile_blocks), dim3(256), 0, s, a);
    return hipGetLastError();
  } else {
    using CF = Cfg<ABITS, false>;
    const int ntiles = ((a.M + CF::BM - 1) / CF::BM) * ((a.N + CF::BN - 1) / CF::BN);
    a.ndp = ntiles;
    a.split = 1;
    a.partial = nullptr;
    hipLaunchKernelGGL((gemm_simple_kernel<ABITS, EPI>), dim3(ntiles), dim3(CF::NTHREADS), 0, s, a);
    return hipGetLastError();
  }
}

// 8-bit activations: 128-wide weight groups take the weight-streaming kernel
// (few tokens) or the pipelined one; one step per output channel (w_group =
// K) the pipelined one with int32 sums over K; other group widths the
// non-pipelined kernel.
// The fp8 4-bit kernel: the same tiles, work list and split tail as the
// 4-bit pipelined kernel.
template <int EPI>
hipError_t launch_a4f8(const GemmArgs& a0, hipStream_t s, float* partial, size_t partial_bytes) {
  GemmArgs a = a0;
  const int slots = device_cus() * 2;
  const Plan p = pipe_plan<4>(a.M, a.N, a.K, partial ? partial_bytes : 0);
  a.ndp = p.ndp;
  a.split = p.split;
  a.partial = p.split > 1 ? partial : nullptr;
  const int rest = p.ntiles - p.ndp;
  const int nitems = p.ndp + rest * p.split;
  hipLaunchKernelGGL((gemm_a4f8_kernel<EPI>), dim3(static_cast<unsigned>(std::min(nitems, slots))), dim3(256), 0, s,
                     a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || rest == 0 || p.split == 1) return e;
  constexpr int per_tile_blocks = F8Layout::BM * F8Layout::BN / 4 / 256;
  hipLaunchKernelGGL((gemm_tail_kernel<4, EPI, false>), dim3(rest * per_tile_blocks), dim3(256), 0, s, a);
  return hipGetLastError();
}

template <int EPI>
hipError_t launch_a8(const GemmArgs& a, hipStream_t s, float* partial, size_t partial_bytes) {
  if (skinny_applies(8, a.M, a.K, a.w_group)) return launch_skinny(8, EPI, a, s, partial, partial_bytes);
  if (a.w_group == KT) return launch_t<8, EPI, true>(a, s, partial, partial_bytes);
  if (a.w_group == a.K) return launch_t<8, EPI, true, true>(a, s, partial, partial_bytes);
  return launch_t<8, EPI, false>(a, s, partial, partial_bytes);
}

}  // namespace

// Compute units of the current device (256 on MI355X; also the fallback when
// there is no device, e.g. for host-only workspace queries), capped at 256.
int device_cus() {
  static std::atomic<int> cache[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  int v = cache[dev].load(std::memory_order_relaxed);
  if (v == 0) {
    int cus = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0) return 256;
    v = std::min(cus, 256);
    cache[dev].store(v, std::memory_order_relaxed);
  }
  return v;
}

size_t gemm_partial_bytes(int act_bits, int32_t M, int32_t N, int32_t K, int32_t w_group) {
  if (act_bits == 8 && w_group != KT && w_group != K) return 0;  // the non-pipelined kernel never splits
  if (skinny_applies(act_bits, M, K, w_group)) return skinny_partial_bytes(act_bits, M, N, K);
  const Plan p = act_bits == 8 ? pipe_plan<8>(M, N, K, ~static_cast<size_t>(0))
                               : pipe_plan<4>(M, N, K, ~static_cast<size_t>(0));
  const size_t unit = static_cast<size_t>(Cfg<8, kPipeWide>::BM) * Cfg<8, kPipeWide>::BN * sizeof(float);
  return static_cast<size_t>(p.ntiles - p.ndp) * (p.split > 1 ? p.split : 0) * unit;
}

hipError_t launch_gemm_gelu_quant(const GemmArgs& a, hipStream_t s, float* partial, size_t partial_bytes) {
  if (skinny_applies(8, a.M, a.K, a.w_group)) return launch_skinny(8, kEpiGelu, a, s, partial, partial_bytes);
  if (a.w_group == a.K) return launch_t<8, kEpiGelu, true, true>(a, s, partial, partial_bytes);  // one step per channel
  if (a.w_group != KT) return hipErrorInvalidValue;
  return launch_t<8, kEpiGelu, true>(a, s, partial, partial_bytes);
}

hipError_t launch_gemm_gelu_quant4(const GemmArgs& a, hipStream_t s, float* partial, size_t partial_bytes) {
  if (skinny_applies(4, a.M, a.K, a.w_group)) return launch_skinny(4, kEpiGelu, a, s, partial, partial_bytes);
  return launch_a4f8<kEpiGelu>(a, s, partial, partial_bytes);
}

hipError_t launch_gemm(int act_bits, int epi, const GemmArgs& a, hipStream_t s, float* partial,
                       size_t partial_bytes) {
  if (act_bits == 8) {
    switch (epi) {
      case kEpiOut: return launch_a8<kEpiOut>(a, s, partial, partial_bytes);
      case kEpiPartial: return launch_a8<kEpiPartial>(a, s, partial, partial_bytes);
      case kEpiInt32: return launch_t<8, kEpiInt32, false>(a, s, nullptr, 0);
      case kEpiDump: return launch_t<8, kEpiDump, false>(a, s, nullptr, 0);
    }
  } else {
    switch (epi) {
      case kEpiOut:
      case kEpiPartial:
        if (a.kc != nullptr)
          return epi == kEpiOut ? launch_a4f8<kEpiOut>(a, s, partial, partial_bytes)
                                : launch_a4f8<kEpiPartial>(a, s, partial, partial_bytes);
        if (skinny_applies(4, a.M, a.K, a.w_group)) return launch_skinny(4, epi, a, s, partial, partial_bytes);
        return epi == kEpiOut ? launch_t<4, kEpiOut, true>(a, s, partial, partial_bytes)
                              : launch_t<4, kEpiPartial, true>(a, s, partial, partial_bytes);
      case kEpiDump: return launch_t<4, kEpiDump, false>(a, s, nullptr, 0);
    }
  }
  return hipErrorInvalidValue;
}

}  // namespace sq
