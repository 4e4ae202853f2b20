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
// the row scale r_i factors out and is applied once in the epilogue) or
// y += (fp32(C) * sigma_i) * Delta_W (4-bit).  The epilogue multiplies by r_i (8-bit) or by
// kappa_i = 1/gamma_s(i) (4-bit, the compensation of Eq. 8), adds the bias and
// casts.
#include <algorithm>
#include <atomic>
#include <type_traits>

#include "sq_internal.h"

namespace sq {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));
typedef __attribute__((address_space(3))) uint8_t lds_u8_t;

constexpr int KT = kKTile;   // 128 channels per stage
constexpr int TM = 2;        // 32-row MFMA tiles per wave
constexpr int TN = 2;        // 32-col MFMA tiles per wave
constexpr int GROUP_M = 8;   // m-tiles per supertile (L2 reuse)

// Workgroup shape: NWM x NWN waves of 64 x 64 outputs; a STAGES-deep LDS ring.
// Two workgroups share a CU (LDS <= 80 KB each), so while one waits at its
// barrier the other's waves keep the SIMDs busy.  The 4-bit path folds a
// block from the previous stage during the current one, which must therefore
// outlive the loads two stages ahead: four stages.
template <int ABITS>
struct Cfg {
  static constexpr int NWM = 2, NWN = 2;
  static constexpr int NWAVE = NWM * NWN;
  static constexpr int NTHREADS = NWAVE * 64;
  static constexpr int BM = 64 * NWM;
  static constexpr int BN = 64 * NWN;
  static constexpr int STAGES = ABITS == 8 ? 3 : 4;
};

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

// LDS byte offset of a __shared__ object.
__device__ __forceinline__ uint32_t lds_offset(const void* p) {
  return static_cast<uint32_t>(reinterpret_cast<uintptr_t>((const lds_u8_t*)p));
}

// One direct global -> LDS load per lane (16 or 4 bytes) from base + voff:
// lane i's data lands at LDS offset `lds` + i * SIZE.  `base` and `lds` must
// be wave-uniform (an SGPR pair and M0); the per-lane part is a 32-bit offset.
// Issued from inline asm so that the compiler, which cannot see which LDS
// bytes such a load writes, does not wait for all of them before every LDS
// read; the kernel waits for them explicitly (wait_vm_and_barrier).  Nothing
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
template <int ABITS>
struct Layout {
  using CF = Cfg<ABITS>;
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

// Epilogue of one 128 x 128 output tile: row factor, bias, cast, then store
// through LDS so that every lane writes 16 contiguous bytes (whole 128-byte
// lines).  Each wave stages 64 rows x 128 bytes (both 32-column tiles for
// 16-bit outputs, one for fp32) in its own region of `smem` (>= 4 x 9 KB, not
// in use by any wave of the workgroup).  Loads of bias and row factors come
// before the stores (as far as the compiler knows the output may alias them).
template <int ABITS, int EPI>
__device__ __forceinline__ void store_tile(const GemmArgs& a, float (&y)[TM][TN][16], int m0, int n0, int wm,
                                           int wn, int wave, int lane, uint8_t* smem) {
  const int M = a.M, N = a.N;
  constexpr int EP_PITCH = 144;  // bytes per staged row (16-byte aligned, spreads banks)
  uint8_t* ep = smem + wave * 64 * EP_PITCH;
  const bool cols_ok = n0 + wn * 64 < N;  // N % 64 == 0: a wave's 64 columns are all in or all out
  float bcol[TN];
#pragma unroll
  for (int tn = 0; tn < TN; ++tn) {
    const int n = min(n0 + wn * 64 + tn * 32 + (lane & 31), N - 1);
    bcol[tn] = (EPI == kEpiOut && a.bias != nullptr) ? bf16_to_f32(a.bias[n]) : 0.0f;
  }
  const int esz = (EPI == kEpiPartial || a.out_dtype == SQ_OUT_F32) ? 4 : 2;
  const int npass = esz == 4 ? 2 : 1;  // fp32: one 32-column tile per pass
#pragma unroll
  for (int tm = 0; tm < TM; ++tm) {
    float rowf[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int m = min(m0 + wm * 64 + tm * 32 + (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3), M - 1);
      rowf[r] = 1.0f;
      if constexpr (EPI == kEpiOut) {
        if constexpr (ABITS == 8) {
          rowf[r] = static_cast<const float*>(a.act_scale)[m];
        } else {
          rowf[r] = 1.0f / a.gamma[a.step * a.S + a.tok2stream[m]];
        }
      }
    }
#pragma unroll
    for (int r = 0; r < 16; ++r)
#pragma unroll
      for (int tn = 0; tn < TN; ++tn) {
        const float v = EPI == kEpiPartial ? y[tm][tn][r] : __builtin_fmaf(y[tm][tn][r], rowf[r], bcol[tn]);
        y[tm][tn][r] = v;
      }
  }
  // constant trip count: `pass` indexes y, which must stay in registers
#pragma unroll
  for (int pass = 0; pass < 2; ++pass) {
    if (pass >= npass) break;
    // stage: row (within the wave's 64) = tm*32 + (r>>2)*8 + (lane>>5)*4 + (r&3)
#pragma unroll
    for (int tm = 0; tm < TM; ++tm)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = tm * 32 + (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3);
        uint8_t* rp = ep + row * EP_PITCH;
        if (esz == 4) {
          reinterpret_cast<float*>(rp)[lane & 31] = y[tm][pass][r];
        } else {
#pragma unroll
          for (int tn = 0; tn < TN; ++tn) {
            const float v = y[tm][tn][r];
            const uint32_t b = a.out_dtype == SQ_OUT_BF16 ? f32_to_bf16(v) : f32_to_f16(v);
            reinterpret_cast<uint16_t*>(rp)[tn * 32 + (lane & 31)] = static_cast<uint16_t>(b);
          }
        }
      }
    // read back 16-byte chunks (8 rows of 128 bytes per instruction) and store
    if (cols_ok) {
      const size_t row_bytes = static_cast<size_t>(N) * esz;
      uint8_t* gbase = static_cast<uint8_t*>(a.out) + static_cast<size_t>(n0 + wn * 64 + pass * 32) * esz;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int row = i * 8 + (lane >> 3);
        const int m = m0 + wm * 64 + row;
        const uint4 v = *reinterpret_cast<const uint4*>(ep + row * EP_PITCH + (lane & 7) * 16);
        if (m < M) *reinterpret_cast<uint4*>(gbase + static_cast<size_t>(m) * row_bytes + (lane & 7) * 16) = v;
      }
    }
  }
}


// ABITS: 8 or 4.  EPI: EpiMode.  W128: 8-bit activations with one weight step
// per 128 input channels (one K-block per pipeline stage).
// PIPE (full or partial epilogue, and either 4-bit activations or W128): the
// overlapped path.  Otherwise blocks are folded (or dumped) when they end.
template <int ABITS, int EPI, bool W128>
__global__ __launch_bounds__(Cfg<ABITS>::NTHREADS, 2) void gemm_w4_kernel(GemmArgs a) {
  using LY = Layout<ABITS>;
  using CF = Cfg<ABITS>;
  constexpr int BM = CF::BM, BN = CF::BN, STAGES = CF::STAGES;
  constexpr bool NEED_SCALE = (EPI == kEpiOut || EPI == kEpiPartial);
  constexpr bool LOAD_SIGMA = ABITS == 4 && NEED_SCALE;
  constexpr bool PIPE = NEED_SCALE && (ABITS == 4 || W128);
  constexpr int NDMA = LY::A_DMA + LY::B_DMA + (LOAD_SIGMA ? 1 : 0) + (NEED_SCALE ? 1 : 0);
  constexpr float WFOLD = ABITS == 8 ? 0.0625f : 0.00390625f;  // 1/16 or 1/256

  __shared__ __align__(1024) uint8_t smem[STAGES * LY::STAGE];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  // wave-uniform (an SGPR): keeps every per-wave LDS and global address scalar
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / CF::NWN, wn = wave % CF::NWN;
  const int h = lane >> 5;
  const int M = a.M, N = a.N, K = a.K;

  const int ntm = (M + BM - 1) / BM;
  const int ntn = (N + BN - 1) / BN;
  const int nkt = K / KT;
  // whole tile, or one K range [kt_begin, kt_end) of a split tail tile
  int lid, kt_begin = 0, kt_end = nkt, unit = -1;
  if (static_cast<int>(blockIdx.x) < a.ndp) {
    lid = xcd_order(blockIdx.x, a.ndp);
  } else {
    unit = blockIdx.x - a.ndp;
    lid = a.ndp + unit / a.split;
    const int sl = unit % a.split;
    kt_begin = sl * nkt / a.split;
    kt_end = (sl + 1) * nkt / a.split;
  }
  int tile_m, tile_n;
  supertile(lid, ntm, ntn, tile_m, tile_n);
  const int m0 = tile_m * BM;
  const int n0 = tile_n * BN;
  const uint8_t* qx = static_cast<const uint8_t*>(a.qx);
  const uint32_t smem_lds = lds_offset(smem);

  // ---- this wave's direct loads: uniform bases (the tile's first row /
  // column, advanced per stage) and 32-bit per-lane offsets within the tile
  const size_t a_row_bytes = ABITS == 8 ? static_cast<size_t>(K) : static_cast<size_t>(K / 2);
  const uint8_t* baseA = qx + static_cast<size_t>(m0) * a_row_bytes;
  const uint8_t* baseB = a.qw + static_cast<size_t>(n0) * (K / 2);
  const uint8_t* baseS = LOAD_SIGMA ? static_cast<const uint8_t*>(a.act_scale) + static_cast<size_t>(m0) * (K / kA4Group) * 2
                                    : nullptr;
  uint32_t voffA[LY::A_DMA];
  uint32_t voffB[LY::B_DMA];
  uint32_t voffS = 0;
  if constexpr (ABITS == 8) {
#pragma unroll
    for (int i = 0; i < LY::A_DMA; ++i) {
      const int row = 8 * (LY::A_DMA * wave + i) + (lane >> 3);
      const int c = (lane & 7) ^ ((row >> 1) & 7);
      voffA[i] = static_cast<uint32_t>((min(m0 + row, M - 1) - m0) * a_row_bytes) + c * 16;
    }
  } else {
#pragma unroll
    for (int i = 0; i < LY::A_DMA; ++i) {
      const int row = 16 * (LY::A_DMA * wave + i) + (lane >> 2);
      const int c = (lane & 3) ^ ((row >> 2) & 3);
      voffA[i] = static_cast<uint32_t>((min(m0 + row, M - 1) - m0) * a_row_bytes) + c * 16;
    }
  }
#pragma unroll
  for (int i = 0; i < LY::B_DMA; ++i) {
    const int col = 16 * (LY::B_DMA * wave + i) + (lane >> 2);
    const int c = (lane & 3) ^ ((col >> 2) & 3);
    voffB[i] = static_cast<uint32_t>((min(n0 + col, N - 1) - n0) * (K / 2)) + c * 16;
  }
  if constexpr (LOAD_SIGMA) {
    const int row = LY::S_ROWS * wave + (lane % LY::S_ROWS);
    voffS = static_cast<uint32_t>((min(m0 + row, M - 1) - m0) * (K / kA4Group) * 2);
  }
  // weight steps: the dword of output channels c, c + 1 of this wave's 64
  // (c even; N is even, so the pair is clamped inside the row)
  const uint32_t wcol2 = static_cast<uint32_t>(min(n0 + wn * 64 + 2 * (lane & 31), N - 2));

  // Loads stage kt into ring slot kt % STAGES.  Past the last stage of the
  // range the source is clamped to that stage: the slot written is free (its
  // stage was consumed before the previous barrier) and is never read again,
  // and the loop body stays free of branches, so its MFMAs and VALU work can
  // be interleaved.
  auto issue_stage = [&](int kt_slot) {
    const uint32_t st = smem_lds + (kt_slot % STAGES) * LY::STAGE;
    const int kt = min(kt_slot, kt_end - 1);
    const uint8_t* bA = baseA + kt * (ABITS == 8 ? KT : KT / 2);
    const uint8_t* bB = baseB + kt * (KT / 2);
#pragma unroll
    for (int i = 0; i < LY::A_DMA; ++i) dma<16>(bA, voffA[i], st + (LY::A_DMA * wave + i) * 1024);
#pragma unroll
    for (int i = 0; i < LY::B_DMA; ++i) dma<16>(bB, voffB[i], st + LY::A_BYTES + (LY::B_DMA * wave + i) * 1024);
    if constexpr (LOAD_SIGMA) dma<4>(baseS + kt * 4, voffS, st + LY::A_BYTES + LY::B_BYTES + wave * 256);
    if constexpr (NEED_SCALE) {
      const uint32_t e = static_cast<uint32_t>((kt * KT) / a.w_group) * static_cast<uint32_t>(N) + wcol2;
      dma<4>(a.w_scale, e * 2, st + LY::A_BYTES + LY::B_BYTES + LY::S_BYTES + wave * 256);
    }
  };

  // ---- per-lane LDS read offsets (within a stage); the swizzle terms depend
  // on the lane only, since every wave's first row and column are multiples
  // of 16, and a 32-row (32-column) step leaves them unchanged: the offsets of
  // the second row (column) tile are the first's plus a constant, which the
  // LDS reads take as an immediate.
  const int arow0 = wm * 64 + (lane & 31);
  const int bcol0 = wn * 64 + (lane & 31);
  constexpr int A_TILE_STEP = ABITS == 8 ? 32 * KT : 32 * (KT / 2);
  constexpr int B_TILE_STEP = 32 * (KT / 2);
  int offA0[4];
#pragma unroll
  for (int ks = 0; ks < 4; ++ks) {
    if constexpr (ABITS == 8)
      offA0[ks] = arow0 * KT + 16 * ((4 * (ks >> 1) + 2 * h + (ks & 1)) ^ ((arow0 >> 1) & 7));
    else
      offA0[ks] = arow0 * (KT / 2) + 16 * ((2 * (ks >> 1) + h) ^ ((arow0 >> 2) & 3));
  }
  int offB0[2];
#pragma unroll
  for (int k2 = 0; k2 < 2; ++k2)
    offB0[k2] = LY::A_BYTES + bcol0 * (KT / 2) + 16 * ((2 * k2 + h) ^ ((bcol0 >> 2) & 3));
  auto offA = [&](int tm, int ks) { return offA0[ks] + tm * A_TILE_STEP; };
  auto offB = [&](int tn, int k2) { return offB0[k2] + tn * B_TILE_STEP; };

  float y[TM][TN][16];
#pragma unroll
  for (int tm = 0; tm < TM; ++tm)
#pragma unroll
    for (int tn = 0; tn < TN; ++tn)
#pragma unroll
      for (int r = 0; r < 16; ++r) y[tm][tn][r] = 0.0f;

  // weight steps of stage kt for the owned columns, widened-code factor folded in
  auto read_wscale = [&](const uint8_t* st, int kt, float (&w)[TN]) {
    const uint32_t* Wst = reinterpret_cast<const uint32_t*>(st + LY::A_BYTES + LY::B_BYTES + LY::S_BYTES + wave * 256);
#pragma unroll
    for (int tn = 0; tn < TN; ++tn) {
      const int c = tn * 32 + (lane & 31);  // column within the wave's 64
      const uint32_t pair = Wst[c >> 1];
      w[tn] = f16_to_f32((c & 1) ? (pair >> 16) : (pair & 0xFFFFu)) * WFOLD;
    }
  };

  // MFMA fragments of k-step ks of a stage.
  auto frags = [&](const uint8_t* st, int ks, v4i (&af)[TM], v4i (&bf)[TN], uint4 (&pa)[TM], uint4 (&pb)[TN]) {
#pragma unroll
    for (int tm = 0; tm < TM; ++tm) {
      if constexpr (ABITS == 8) {
        af[tm] = *reinterpret_cast<const v4i*>(st + offA(tm, ks));
      } else {
        if ((ks & 1) == 0) pa[tm] = *reinterpret_cast<const uint4*>(st + offA(tm, ks));
        af[tm] = (ks & 1) ? unpack_frag(pa[tm].z, pa[tm].w) : unpack_frag(pa[tm].x, pa[tm].y);
      }
    }
#pragma unroll
    for (int tn = 0; tn < TN; ++tn) {
      if ((ks & 1) == 0) pb[tn] = *reinterpret_cast<const uint4*>(st + offB(tn, ks >> 1));
      bf[tn] = (ks & 1) ? unpack_frag(pb[tn].z, pb[tn].w) : unpack_frag(pb[tn].x, pb[tn].y);
    }
  };

  // y += fp32(C) * Delta_W for one 32 x 32 tile (8-bit activations)
  auto fold8 = [&](const v16i& c, float w, float (&yt)[16]) {
#pragma unroll
    for (int r = 0; r < 16; ++r) yt[r] = __builtin_fmaf(static_cast<float>(c[r]), w, yt[r]);
  };
  // y += (fp32(C) * sigma_row) * Delta_W for row-tile tm and both column
  // tiles (4-bit activations); sigma from stage `st`, block half hb
  auto fold4 = [&](const uint8_t* st, int hb, const v16i (&c)[TN], int tm, const float (&w)[TN], bool valid) {
    const uint8_t* S = st + LY::A_BYTES + LY::B_BYTES;
#pragma unroll
    for (int r4 = 0; r4 < 4; ++r4) {
      const int ml = wm * 64 + tm * 32 + r4 * 8 + (lane >> 5) * 4;
      const uint4 sp = *reinterpret_cast<const uint4*>(S + (ml / LY::S_ROWS) * 256 + (ml % LY::S_ROWS) * 4);
      const uint32_t w4[4] = {sp.x, sp.y, sp.z, sp.w};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float sg = valid ? f16_to_f32(hb ? (w4[i] >> 16) : (w4[i] & 0xFFFFu)) : 0.0f;
#pragma unroll
        for (int tn = 0; tn < TN; ++tn) {
          const int r = r4 * 4 + i;
          y[tm][tn][r] = __builtin_fmaf(static_cast<float>(c[tn][r]) * sg, w[tn], y[tm][tn][r]);
        }
      }
    }
  };

  issue_stage(kt_begin);
  issue_stage(kt_begin + 1);
  wait_vm_and_barrier<NDMA>();

  if constexpr (PIPE && ABITS == 8) {
    // ---------------- 8-bit activations, one block per stage.  Tile-major:
    // for each 32 x 32 tile, fold the previous block's accumulator into y,
    // then run the tile's four MFMAs of this block; the fold of the next tile
    // (VALU) overlaps these MFMAs.
    // zero accumulators and steps: the fold before the first block adds 0
    v16i acc[TM][TN];
    float wsv_prev[TN], wsv[TN];
#pragma unroll
    for (int tm = 0; tm < TM; ++tm)
#pragma unroll
      for (int tn = 0; tn < TN; ++tn) acc[tm][tn] = (v16i)(0);
#pragma unroll
    for (int tn = 0; tn < TN; ++tn) wsv_prev[tn] = 0.0f;
    for (int kt = kt_begin; kt < kt_end; ++kt) {
      issue_stage(kt + 2);
      const uint8_t* st = smem + (kt % STAGES) * LY::STAGE;
      read_wscale(st, kt, wsv);
      v4i bfull[TN][4];
#pragma unroll
      for (int tn = 0; tn < TN; ++tn)
#pragma unroll
        for (int k2 = 0; k2 < 2; ++k2) {
          const uint4 pb = *reinterpret_cast<const uint4*>(st + offB(tn, k2));
          bfull[tn][2 * k2] = unpack_frag(pb.x, pb.y);
          bfull[tn][2 * k2 + 1] = unpack_frag(pb.z, pb.w);
        }
#pragma unroll
      for (int tm = 0; tm < TM; ++tm) {
        v4i af[4];
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) af[ks] = *reinterpret_cast<const v4i*>(st + offA(tm, ks));
#pragma unroll
        for (int tn = 0; tn < TN; ++tn) {
          fold8(acc[tm][tn], wsv_prev[tn], y[tm][tn]);
          acc[tm][tn] = __builtin_amdgcn_mfma_i32_32x32x32_i8(af[0], bfull[tn][0], (v16i)(0), 0, 0, 0);
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
      wait_vm_and_barrier<NDMA>();
    }
#pragma unroll
    for (int t = 0; t < TM * TN; ++t) fold8(acc[t >> 1][t & 1], wsv_prev[t & 1], y[t >> 1][t & 1]);
  } else if constexpr (PIPE && ABITS == 4) {
    // ---------------- 4-bit activations: blocks are the two halves of a
    // stage.  Row-tile-major: fold the previous block's accumulators of a
    // row tile (they share its group steps), then run its MFMAs of this block.
    // zero accumulators and steps: the fold before the first block adds 0
    v16i acc[TM][TN];
    float wsv_prev[TN], wsv[TN];
#pragma unroll
    for (int tm = 0; tm < TM; ++tm)
#pragma unroll
      for (int tn = 0; tn < TN; ++tn) acc[tm][tn] = (v16i)(0);
#pragma unroll
    for (int tn = 0; tn < TN; ++tn) wsv_prev[tn] = 0.0f;
    for (int kt = kt_begin; kt < kt_end; ++kt) {
      issue_stage(kt + 2);
      const uint8_t* st = smem + (kt % STAGES) * LY::STAGE;
      const uint8_t* st_prev = smem + ((kt + STAGES - 1) % STAGES) * LY::STAGE;
      read_wscale(st, kt, wsv);
#pragma unroll
      for (int hb = 0; hb < 2; ++hb) {
        v4i bf[TN][2];
#pragma unroll
        for (int tn = 0; tn < TN; ++tn) {
          const uint4 pb = *reinterpret_cast<const uint4*>(st + offB(tn, hb));
          bf[tn][0] = unpack_frag(pb.x, pb.y);
          bf[tn][1] = unpack_frag(pb.z, pb.w);
        }
#pragma unroll
        for (int tm = 0; tm < TM; ++tm) {
          const uint4 pa = *reinterpret_cast<const uint4*>(st + offA(tm, 2 * hb));
          const v4i af0 = unpack_frag(pa.x, pa.y);
          const v4i af1 = unpack_frag(pa.z, pa.w);
          // previous block: second half of the previous stage, or first half of this one
          if (hb == 0) {
            fold4(st_prev, 1, acc[tm], tm, wsv_prev, kt > kt_begin);
          } else {
            fold4(st, 0, acc[tm], tm, wsv, true);
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
      wait_vm_and_barrier<NDMA>();
    }
    {
      const uint8_t* st_last = smem + ((kt_end - 1) % STAGES) * LY::STAGE;
#pragma unroll
      for (int tm = 0; tm < TM; ++tm) fold4(st_last, 1, acc[tm], tm, wsv_prev, true);
    }
  } else {
    // ---------------- blocks folded or dumped when they end
    v16i acc[TM][TN];
#pragma unroll
    for (int tm = 0; tm < TM; ++tm)
#pragma unroll
      for (int tn = 0; tn < TN; ++tn) acc[tm][tn] = (v16i)(0);
    for (int kt = 0; kt < nkt; ++kt) {
      issue_stage(kt + 2);
      const uint8_t* st = smem + (kt % STAGES) * LY::STAGE;
      float wsv[TN];
      if constexpr (NEED_SCALE) read_wscale(st, kt, wsv);
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
        frags(st, ks, af, bf, pa, pb);
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
            for (int t = 0; t < TM * TN; ++t) fold8(acc[t >> 1][t & 1], wsv[t & 1], y[t >> 1][t & 1]);
          }
        }
      }
      wait_vm_and_barrier<NDMA>();
    }
    if constexpr (EPI == kEpiInt32) dump_block<ABITS>(a, acc, 0, m0, n0, wm, wn, lane);
  }

  // drain the clamped loads issued by the last iterations before the LDS is
  // reused (or the workgroup ends)
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  if constexpr (!NEED_SCALE) return;
  if constexpr (PIPE) {
    if (unit >= 0) {
      // split tail: this K range's fp32 sums of the tile, row-major [BM][BN]
      float* P = a.partial + static_cast<size_t>(unit) * BM * BN;
#pragma unroll
      for (int tm = 0; tm < TM; ++tm)
#pragma unroll
        for (int tn = 0; tn < TN; ++tn)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int row = wm * 64 + tm * 32 + (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3);
            P[row * BN + wn * 64 + tn * 32 + (lane & 31)] = y[tm][tn][r];
          }
      return;
    }
  }

  __syncthreads();
  store_tile<ABITS, EPI>(a, y, m0, n0, wm, wn, wave, lane, smem);
}

// Second kernel of a split tail: adds the `split` partial sums of every
// output of the split tiles in range order (so the result does not depend on
// which range finished first) and finishes it exactly as store_tile does
// (one fma with the row factor and the bias, then the cast).  Four adjacent
// outputs per thread, 16-byte loads.
template <int ABITS, int EPI>
__global__ __launch_bounds__(256) void gemm_tail_kernel(GemmArgs a) {
  constexpr int BM = Cfg<ABITS>::BM, BN = Cfg<ABITS>::BN;
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
  float4 acc = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
#pragma unroll 8
  for (int sl = 0; sl < a.split; ++sl) {
    const float4 v = *reinterpret_cast<const float4*>(P + static_cast<size_t>(sl) * BM * BN);
    acc.x += v.x;
    acc.y += v.y;
    acc.z += v.z;
    acc.w += v.w;
  }
  float y[4] = {acc.x, acc.y, acc.z, acc.w};
  if constexpr (EPI == kEpiOut) {
    const float rowf = ABITS == 8 ? static_cast<const float*>(a.act_scale)[m]
                                  : 1.0f / a.gamma[a.step * a.S + a.tok2stream[m]];
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
    uint32_t h[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) h[j] = a.out_dtype == SQ_OUT_BF16 ? f32_to_bf16(y[j]) : f32_to_f16(y[j]);
    *reinterpret_cast<uint2*>(static_cast<uint16_t*>(a.out) + static_cast<size_t>(m) * a.N + n) =
        make_uint2(h[0] | (h[1] << 16), h[2] | (h[3] << 16));
  }
}

// Workgroups that fit on the device at once (two per CU), capped at 512.
int device_slots() {
  static std::atomic<int> cache[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 512;
  int v = cache[dev].load(std::memory_order_relaxed);
  if (v == 0) {
    int cus = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0) return 512;
    v = std::min(2 * cus, 512);
    cache[dev].store(v, std::memory_order_relaxed);
  }
  return v;
}

constexpr size_t kUnitBytes = 128 * 128 * sizeof(float);  // partial sums of one tile range

// Split plan: the tiles that fill whole rounds of `slots` run whole; each of
// the R left over is split into S >= 2 K ranges of >= 2 stages (S * R <=
// slots / 2 when whole rounds run, <= slots otherwise), if `partial_bytes`
// holds R * S units.  Only the pipelined paths split (their blocks never
// straddle a range boundary).
struct Plan {
  int ntiles, ndp, split;
};
Plan plan_split(int act_bits, int epi, int32_t M, int32_t N, int32_t K, int32_t w_group, int slots,
                size_t partial_bytes) {
  const int ntiles = ((M + 127) / 128) * ((N + 127) / 128);
  Plan p{ntiles, ntiles, 1};
  const bool pipe = (epi == kEpiOut || epi == kEpiPartial) && (act_bits == 4 || w_group == KT);
  const int nkt = K / KT;
  const int rest = ntiles % slots;
  if (!pipe || rest == 0 || nkt < 4) return p;
  int split = std::min(nkt / 2, ntiles >= slots ? slots / rest / 2 : slots / rest);
  while (split >= 2 && static_cast<size_t>(rest) * split * kUnitBytes > partial_bytes) --split;
  if (split < 2) return p;
  p.ndp = ntiles - rest;
  p.split = split;
  return p;
}

template <int ABITS, int EPI, bool W128>
hipError_t launch_t(const GemmArgs& a0, hipStream_t s, float* partial, size_t partial_bytes) {
  GemmArgs a = a0;
  const Plan p = plan_split(ABITS, EPI, a.M, a.N, a.K, a.w_group, device_slots(), partial ? partial_bytes : 0);
  a.ndp = p.ndp;
  a.split = p.split;
  a.partial = p.split > 1 ? partial : nullptr;
  const int rest = p.ntiles - p.ndp;
  const unsigned grid = static_cast<unsigned>(p.ndp + rest * p.split);
  hipLaunchKernelGGL((gemm_w4_kernel<ABITS, EPI, W128>), dim3(grid), dim3(Cfg<ABITS>::NTHREADS), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || rest == 0 || p.split == 1) return e;
  if constexpr (EPI == kEpiOut || EPI == kEpiPartial) {
    constexpr int per_tile_blocks = Cfg<ABITS>::BM * Cfg<ABITS>::BN / 4 / 256;
    hipLaunchKernelGGL((gemm_tail_kernel<ABITS, EPI>), dim3(rest * per_tile_blocks), dim3(256), 0, s, a);
    return hipGetLastError();
  }
  return hipErrorInvalidValue;
}

template <int EPI>
hipError_t launch_a8(const GemmArgs& a, hipStream_t s, float* partial, size_t partial_bytes) {
  return a.w_group == KT ? launch_t<8, EPI, true>(a, s, partial, partial_bytes)
                         : launch_t<8, EPI, false>(a, s, partial, partial_bytes);
}

}  // namespace

size_t gemm_partial_bytes(int act_bits, int32_t M, int32_t N, int32_t K, int32_t w_group) {
  const Plan p = plan_split(act_bits, kEpiOut, M, N, K, w_group, device_slots(), ~static_cast<size_t>(0));
  return static_cast<size_t>(p.ntiles - p.ndp) * (p.split > 1 ? p.split : 0) * kUnitBytes;
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
      case kEpiOut: return launch_t<4, kEpiOut, false>(a, s, partial, partial_bytes);
      case kEpiPartial: return launch_t<4, kEpiPartial, false>(a, s, partial, partial_bytes);
      case kEpiDump: return launch_t<4, kEpiDump, false>(a, s, nullptr, 0);
    }
  }
  return hipErrorInvalidValue;
}

}  // namespace sq
