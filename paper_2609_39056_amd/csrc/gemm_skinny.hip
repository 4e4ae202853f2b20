// Weight-streaming GEMM for few tokens (the second fused kernel of Sec. 4.4
// when a layer runs the action and proprioception streams alone, at most 128
// tokens): the operands, block accumulation and epilogue of the tiled kernel.
#include <algorithm>

#include "gelu.h"
#include "gemm_frag.h"
#include "sq_internal.h"

namespace sq {
namespace {


// The work is streaming the weights.  A workgroup owns 64 rows x 32 output
// channels over a range of K; its four waves take alternate stages of that
// range and keep their own fp32 sums, added through LDS in wave order at the
// end, each wave then finishing a quarter of the outputs.  Every byte of a
// stage (activation codes, 4-bit group steps, packed weights, weight steps)
// is copied by direct global -> LDS loads into the wave's own ring of LDS
// slots, loaded two stages ahead: whole cache lines per instruction, so the
// activation rows that every workgroup reads cost little on the vector memory
// path.  Each wave reads only what it loaded itself, so the main loop waits on
// its own load counter and has no barriers.  When the output channels alone
// give too few workgroups, K is also split across workgroups: each leaves
// fp32 sums of its 64 x 32 outputs, which a second kernel adds in range order.
// With one weight step per output channel (PC: w_group = K, 8-bit
// activations) there is no fold in the loop: each wave keeps int32 sums over
// its stages, the four are added in integers, and the total is converted and
// scaled once (split ranges hand int32 sums to the second kernel).
// t rounded to the nearest integer, ties to even (abs(t) <= 2^22): the low
// byte of t + 1.5 * 2^23 is the two's-complement code.
__device__ __forceinline__ uint32_t rne_code_bits8(float t) { return __float_as_uint(t + 12582912.0f); }
// The low bytes of four words, in order, as one word.
__device__ __forceinline__ uint32_t pack_bytes8(uint32_t w0, uint32_t w1, uint32_t w2, uint32_t w3) {
  const uint32_t lo = __builtin_amdgcn_perm(w1, w0, 0x0c0c0400u);
  const uint32_t hi = __builtin_amdgcn_perm(w3, w2, 0x0c0c0400u);
  return __builtin_amdgcn_perm(hi, lo, 0x05040100u);
}

// Rows per workgroup: 64 (two 32-row MFMA tiles per wave), or 32 when the
// 64-row blocks would leave CUs without a workgroup (few output channels,
// e.g. the 2048-wide out and down projections): half the rows per workgroup
// and half its LDS, so that twice as many workgroups run, two per CU.
// Output channels per workgroup: 32, or 64 when 32-channel strips would need
// more than one round of workgroups (the 128-token 2B projections, the 14B
// ones at 64 tokens): each wave then computes two 32-channel tiles with the
// same activation fragments.
constexpr int SK_BM = 64;
constexpr int SK_BN = 32;
constexpr int SK_DIST = 2;  // stages loaded ahead (the codes kernels)

// LDS layout of a slot (16-byte chunks XOR-swizzled, as in the tiled kernel,
// so that fragment reads are free of bank conflicts):
//   8-bit activation row r (128 B) at r * 128, chunk c at position c ^ ((r >> 1) & 7)
//   4-bit activation row r (64 B) at r * 64, chunk c at position c ^ ((r >> 2) & 3)
//   weight column n (64 B, n < BN) at B_OFF + n * 64, chunk c at position c ^ ((n >> 2) & 3)
//   4-bit group steps at S_OFF: row r's dword (the stage's two fp16 steps) at r * 4
//   weight steps at W_OFF: dword i holds columns 2i, 2i + 1
// Lane (column n = 32 tn + (lane & 31) of tile tn, h = lane >> 5) feeds k-step
// s of a stage with the channels [64 (s >> 1) + 32 h + 16 (s & 1), +16) of both
// operands; 64-wide blocks are k-steps {0, 1} and {2, 3}.
// QX (the single-kernel linear, 8-bit STATIC ranges): the slot's activation
// area holds the stage's bf16 rows (row r, 256 B, chunk c at position
// c ^ (r & 15)), which the wave quantizes in place into the 8-bit layout
// above (the first 8 KB) before its MFMAs; one stage is loaded ahead.
template <int ABITS, bool QX = false, int BM = SK_BM, int BN = SK_BN>
struct Sk {
  static constexpr int DIST = QX ? 1 : SK_DIST;  // stages loaded ahead
  static constexpr int SLOTS = DIST + 1;         // ring slots per wave
  static constexpr int A = BM * (QX ? 2 * KT : (ABITS == 8 ? KT : KT / 2));  // bf16 rows, or codes (BM = 64: 8 / 4 KB)
  static constexpr int B = BN * (KT / 2);                       // packed weights (2 or 4 KB)
  static constexpr int SIG = ABITS == 4 ? 256 : 0;              // 4-bit group steps
  static constexpr int B_OFF = A, S_OFF = A + B, W_OFF = A + B + SIG;
  static constexpr int D_OFF = W_OFF + 256;                     // QX: the stage's 128 D^-1 values
  static constexpr int SLOT = D_OFF + (QX ? 512 : 0);           // + one 256 B load of weight steps
  static constexpr int NDMA = A / 1024 + B / 1024 + (ABITS == 4 ? 1 : 0) + 1;  // loads per stage and wave
  static constexpr int WGS_PER_CU = 4 * SLOTS * SLOT * 2 <= 160 * 1024 ? 2 : 1;
  static_assert(4 * SLOTS * SLOT <= 160 * 1024, "the ring fits in the LDS");
  static_assert(4 * BM * BN * 4 <= 4 * SLOTS * SLOT, "the wave sums fit in the ring");
  static_assert(BM == 64 || (BM == 32 && !QX), "64-row blocks, or 32 without in-kernel quantization");
  static_assert(BN == 32 || (BN == 64 && !QX), "64-channel strips without in-kernel quantization");
  static_assert(!QX || ABITS == 8, "in-kernel quantization: 8-bit codes");
};

template <int ABITS, int EPI, bool PC, bool QX = false, int BM = SK_BM, int BN = SK_BN>
__global__ __launch_bounds__(256, (Sk<ABITS, QX, BM, BN>::WGS_PER_CU)) void gemm_skinny_kernel(GemmArgs a) {
  using L = Sk<ABITS, QX, BM, BN>;
  constexpr int TM = BM / 32;  // 32-row MFMA tiles per wave
  constexpr int TN = BN / 32;  // 32-channel MFMA tiles per wave
  static_assert(!PC || ABITS == 8, "one weight step per channel: 8-bit activations");
  static_assert(!QX || EPI == kEpiOut, "the single-kernel linear finishes its outputs");
  __shared__ __attribute__((aligned(16))) uint8_t ring[4][L::SLOTS][L::SLOT];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int M = a.M, N = a.N, K = a.K;
  const int nkt = K / KT;
  const int S = a.split;
  const int strip = blockIdx.x / S, range = blockIdx.x % S;
  const int m0 = blockIdx.y * BM, n0 = strip * BN;
  const int kt0 = range * nkt / S, kt1 = (range + 1) * nkt / S;
  const int h = lane >> 5, col = lane & 31;
  const int rows = min(M - m0, BM);
  const int arow = QX ? 2 * K : (ABITS == 8 ? K : K / 2);  // bytes of an activation row (QX: bf16)

  // direct-load sources: rows past the matrix read its last row
  uint32_t voffA[L::A / 1024];
#pragma unroll
  for (int i = 0; i < L::A / 1024; ++i) {
    if constexpr (QX) {
      const int r = 4 * i + (lane >> 4);
      voffA[i] = static_cast<uint32_t>(min(r, rows - 1) * arow + 16 * ((lane & 15) ^ (r & 15)));
    } else if constexpr (ABITS == 8) {
      const int r = 8 * i + (lane >> 3);
      voffA[i] = static_cast<uint32_t>(min(r, rows - 1) * arow + 16 * ((lane & 7) ^ ((r >> 1) & 7)));
    } else {
      const int r = 16 * i + (lane >> 2);
      voffA[i] = static_cast<uint32_t>(min(r, rows - 1) * arow + 16 * ((lane & 3) ^ ((r >> 2) & 3)));
    }
  }
  uint32_t voffB[L::B / 1024];
#pragma unroll
  for (int i = 0; i < L::B / 1024; ++i) {
    const int n = 16 * i + (lane >> 2);
    voffB[i] = static_cast<uint32_t>(n * (K / 2) + 16 * ((lane & 3) ^ ((n >> 2) & 3)));
  }
  const uint32_t voffS = static_cast<uint32_t>(min(lane, rows - 1) * (K / kA4Group) * 2);  // row lane
  const uint32_t voffW = 4 * (lane & (BN / 2 - 1));  // lanes past BN / 2 repeat the first dwords
  const uint32_t ring0 = lds_offset(&ring[wave][0][0]);
  const uint8_t* qx = static_cast<const uint8_t*>(a.qx) + static_cast<size_t>(m0) * arow;
  const uint8_t* qw = a.qw + static_cast<size_t>(n0) * (K / 2);
  const uint16_t* sig = static_cast<const uint16_t*>(a.act_scale) + static_cast<size_t>(m0) * (K / kA4Group);
  auto issue = [&](int kt, int slot) {
    const uint32_t st = ring0 + slot * L::SLOT;
#pragma unroll
    for (int i = 0; i < L::A / 1024; ++i) dma<16>(qx + kt * (arow / nkt), voffA[i], st + i * 1024);
#pragma unroll
    for (int i = 0; i < L::B / 1024; ++i) dma<16>(qw + kt * (KT / 2), voffB[i], st + L::B_OFF + i * 1024);
    if constexpr (ABITS == 4) dma<4>(sig + 2 * kt, voffS, st + L::S_OFF);  // the stage's two groups
    // group-major steps of the stage's weight group
    dma<4>(a.w_scale + static_cast<size_t>((kt * KT) / a.w_group) * N + n0, voffW, st + L::W_OFF);
    if constexpr (QX) {  // D^-1 of the stage's channels (one stage ahead: the wait is for all loads)
      if (a.dinv != nullptr) {
        dma<4>(a.dinv + kt * KT, 4 * lane, st + L::D_OFF);
        dma<4>(a.dinv + kt * KT + 64, 4 * lane, st + L::D_OFF + 256);
      }
    }
  };

  // fragment offsets within a slot: activations per (row tile, k-step) for
  // 8-bit, per (row tile, k-step pair) for packed 4-bit rows
  int aoff[TM][4];
#pragma unroll
  for (int tm = 0; tm < TM; ++tm) {
    const int r = tm * 32 + col;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      if constexpr (ABITS == 8)
        aoff[tm][ks] = r * 128 + 16 * ((4 * (ks >> 1) + 2 * h + (ks & 1)) ^ ((r >> 1) & 7));
      else
        aoff[tm][ks] = r * 64 + 16 * ((2 * (ks >> 1) + h) ^ ((r >> 2) & 3));
    }
  }
  int boff[TN][2], woff[TN];
#pragma unroll
  for (int tn = 0; tn < TN; ++tn) {
#pragma unroll
    for (int k2 = 0; k2 < 2; ++k2)
      boff[tn][k2] = L::B_OFF + (32 * tn + col) * 64 + 16 * ((2 * k2 + h) ^ ((col >> 2) & 3));
    woff[tn] = L::W_OFF + 4 * ((32 * tn + col) >> 1);
  }

  float y[TM][TN][16];
  v16i acc[TM][TN];
  float wprev[TN];  // 8-bit: the fold before the first block adds 0
#pragma unroll
  for (int tn = 0; tn < TN; ++tn) {
    wprev[tn] = 0.0f;
#pragma unroll
    for (int tm = 0; tm < TM; ++tm) {
      acc[tm][tn] = (v16i)(0);
#pragma unroll
      for (int r = 0; r < 16; ++r) y[tm][tn][r] = 0.0f;
    }
  }

  // 8-bit: y += fp32(C) * Delta_W of the previous block, then this block's
  // MFMAs.  4-bit: the MFMAs of both 64-blocks of the stage, then their folds
  // with the row group steps and the stage's weight step.
  auto compute = [&](int slot) {
    const uint8_t* st = &ring[wave][slot][0];
    // every LDS read of the stage first: one latency per stage
    uint4 pb[TN][2];
    uint32_t wpair[TN];
    v4i af[TM][4];
#pragma unroll
    for (int tn = 0; tn < TN; ++tn) {
#pragma unroll
      for (int k2 = 0; k2 < 2; ++k2) pb[tn][k2] = *reinterpret_cast<const uint4*>(st + boff[tn][k2]);
      wpair[tn] = *reinterpret_cast<const uint32_t*>(st + woff[tn]);
    }
#pragma unroll
    for (int tm = 0; tm < TM; ++tm)
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        if constexpr (ABITS == 8) {
          af[tm][ks] = *reinterpret_cast<const v4i*>(st + aoff[tm][ks]);
        } else if ((ks & 1) == 0) {
          const uint4 pa = *reinterpret_cast<const uint4*>(st + aoff[tm][ks]);
          af[tm][ks] = __builtin_bit_cast(v4i, pa);  // packed: widened below
        }
      }
    uint4 sp[TM][4];  // 4-bit: group steps of the lane's 16 rows per tile
    if constexpr (ABITS == 4) {
#pragma unroll
      for (int tm = 0; tm < TM; ++tm)
#pragma unroll
        for (int g = 0; g < 4; ++g)
          sp[tm][g] = *reinterpret_cast<const uint4*>(st + L::S_OFF + (tm * 32 + 8 * g + 4 * h) * 4);
    }
    __builtin_amdgcn_sched_barrier(0);
    v4i bf[TN][4];
    float wstep[TN];
#pragma unroll
    for (int tn = 0; tn < TN; ++tn) {
#pragma unroll
      for (int k2 = 0; k2 < 2; ++k2) {
        bf[tn][2 * k2] = unpack_frag(pb[tn][k2].x, pb[tn][k2].y);
        bf[tn][2 * k2 + 1] = unpack_frag(pb[tn][k2].z, pb[tn][k2].w);
      }
      wstep[tn] = f16_to_f32((col & 1) ? (wpair[tn] >> 16) : (wpair[tn] & 0xFFFFu));
    }
    if constexpr (PC) {
#pragma unroll
      for (int tm = 0; tm < TM; ++tm)
#pragma unroll
        for (int tn = 0; tn < TN; ++tn)
#pragma unroll
          for (int ks = 0; ks < 4; ++ks)
            acc[tm][tn] = __builtin_amdgcn_mfma_i32_32x32x32_i8(af[tm][ks], bf[tn][ks], acc[tm][tn], 0, 0, 0);
    } else if constexpr (ABITS == 8) {
#pragma unroll
      for (int tm = 0; tm < TM; ++tm)
#pragma unroll
        for (int tn = 0; tn < TN; ++tn) {
          fold8(acc[tm][tn], wprev[tn], y[tm][tn]);
          acc[tm][tn] = __builtin_amdgcn_mfma_i32_32x32x32_i8(af[tm][0], bf[tn][0], (v16i)(0), 0, 0, 0);
#pragma unroll
          for (int ks = 1; ks < 4; ++ks)
            acc[tm][tn] = __builtin_amdgcn_mfma_i32_32x32x32_i8(af[tm][ks], bf[tn][ks], acc[tm][tn], 0, 0, 0);
        }
#pragma unroll
      for (int tn = 0; tn < TN; ++tn) wprev[tn] = wstep[tn] * 0.0625f;  // widened weight codes carry a factor 16
    } else {
      v16i c[2][TM][TN];
#pragma unroll
      for (int hb = 0; hb < 2; ++hb)
#pragma unroll
        for (int tm = 0; tm < TM; ++tm) {
          const uint4 pa = __builtin_bit_cast(uint4, af[tm][2 * hb]);
          const v4i a0 = unpack_frag(pa.x, pa.y), a1 = unpack_frag(pa.z, pa.w);
#pragma unroll
          for (int tn = 0; tn < TN; ++tn) {
            c[hb][tm][tn] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a0, bf[tn][2 * hb], (v16i)(0), 0, 0, 0);
            c[hb][tm][tn] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a1, bf[tn][2 * hb + 1], c[hb][tm][tn], 0, 0, 0);
          }
        }
      // block by block, as the tiled kernels: y += (fp32(C_b) sigma_b) * Delta_W
#pragma unroll
      for (int tn = 0; tn < TN; ++tn) {
        const float w = wstep[tn] * 0.00390625f;  // widened codes of both operands carry 16 * 16
#pragma unroll
        for (int tm = 0; tm < TM; ++tm)
#pragma unroll
          for (int g = 0; g < 4; ++g) {
            const uint32_t s4[4] = {sp[tm][g].x, sp[tm][g].y, sp[tm][g].z, sp[tm][g].w};
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              const int r = 4 * g + q;
              y[tm][tn][r] =
                  __builtin_fmaf(mul_step16<0>(static_cast<float>(c[0][tm][tn][r]), s4[q]), w, y[tm][tn][r]);
              y[tm][tn][r] =
                  __builtin_fmaf(mul_step16<1>(static_cast<float>(c[1][tm][tn][r]), s4[q]), w, y[tm][tn][r]);
            }
          }
      }
    }
  };

  // QX: the STATIC quantization of Eq. 1 with the channel scaling of Eq. 6
  // and the gain of Eq. 8, with the first kernel's fp32 chain
  // (q = rint(clamp((x * dinv) * g * (1 / Delta))), Delta = c / 127): lane l
  // quantizes row l of the stage (rows past M repeat the last row)
  float qg = 0.0f, qinv = 0.0f, qdelta = 0.0f;
  if constexpr (QX) {
    qg = a.gamma[a.step * a.S + a.tok2stream[m0 + min(lane, rows - 1)]];
    qdelta = a.clip[a.step] / 127.0f;
    qinv = 1.0f / qdelta;
    if (__builtin_isinf(qinv)) qinv = 0.0f;
  }
  auto quantize = [&](int slot, int kt) {
    uint8_t* st = &ring[wave][slot][0];
    const int r = lane;
    uint4 xv[16];  // the row's 128 bf16 values of the stage, chunk c at position c ^ (r & 15)
#pragma unroll
    for (int c = 0; c < 16; ++c) xv[c] = *reinterpret_cast<const uint4*>(st + r * 256 + 16 * (c ^ (r & 15)));
    const bool has_d = a.dinv != nullptr;
    uint4 out[8];
#pragma unroll
    for (int c16 = 0; c16 < 8; ++c16) {
      // D^-1 of the 16 channels (the same for every lane: broadcast reads);
      // without D, 1 (x * 1 = x exactly)
      float dvv[16];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float4 d4 = *reinterpret_cast<const float4*>(st + L::D_OFF + 64 * c16 + 16 * q);
        dvv[4 * q] = has_d ? d4.x : 1.0f;
        dvv[4 * q + 1] = has_d ? d4.y : 1.0f;
        dvv[4 * q + 2] = has_d ? d4.z : 1.0f;
        dvv[4 * q + 3] = has_d ? d4.w : 1.0f;
      }
      uint32_t b[16];
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int k = 16 * c16 + e;
        const uint32_t w = (k & 7) < 2 ? xv[k >> 3].x : (k & 7) < 4 ? xv[k >> 3].y : (k & 7) < 6 ? xv[k >> 3].z
                                                                                                 : xv[k >> 3].w;
        const float x = __uint_as_float((k & 1) ? (w & 0xFFFF0000u) : (w << 16)) * dvv[e];
        float t = (x * qg) * qinv;
        t = fminf(fmaxf(t, -127.0f), 127.0f);
        b[e] = rne_code_bits8(t);
      }
      out[c16] = make_uint4(pack_bytes8(b[0], b[1], b[2], b[3]), pack_bytes8(b[4], b[5], b[6], b[7]),
                            pack_bytes8(b[8], b[9], b[10], b[11]), pack_bytes8(b[12], b[13], b[14], b[15]));
    }
    // in place: every read of the wave was issued before these writes, and
    // the LDS executes a wave's operations in order
#pragma unroll
    for (int c16 = 0; c16 < 8; ++c16)
      *reinterpret_cast<uint4*>(st + r * KT + 16 * (c16 ^ ((r >> 1) & 7))) = out[c16];
  };

  // this wave's stages kt0 + wave + 4j, j < nst; past the end the last stage
  // is loaded again, so every wait leaves the same number of loads in flight
  const int nst = kt1 - kt0 > wave ? (kt1 - kt0 - wave + 3) / 4 : 0;
  auto stage = [&](int j) { return kt0 + wave + 4 * min(j, nst - 1); };
  if (nst > 0) {
#pragma unroll
    for (int p = 0; p < L::DIST; ++p) issue(stage(p), p);
    for (int j = 0; j < nst; ++j) {
      wait_vm<L::NDMA * (L::DIST - 1)>();                     // stage j has landed
      issue(stage(j + L::DIST), (j + L::DIST) % L::SLOTS);  // into the slot read last iteration
      if constexpr (QX) quantize(j % L::SLOTS, stage(j));
      compute(j % L::SLOTS);
    }
  }
  if constexpr (ABITS == 8 && !PC) {
#pragma unroll
    for (int tm = 0; tm < TM; ++tm)
#pragma unroll
      for (int tn = 0; tn < TN; ++tn) fold8(acc[tm][tn], wprev[tn], y[tm][tn]);
  }

  // the four waves' sums, added in wave order; wave g then finishes register
  // group g of every tile: rows tm * 32 + 8 g + 4 h + q, q < 4
  wait_vm<0>();     // no direct load still writes the ring
  __syncthreads();  // and no wave still reads it
  constexpr int NT = TM * TN;
  float* red = reinterpret_cast<float*>(&ring[0][0][0]);  // [wave][(tm * TN + tn) * 16 + r][lane]
#pragma unroll
  for (int tm = 0; tm < TM; ++tm)
#pragma unroll
    for (int tn = 0; tn < TN; ++tn)
#pragma unroll
      for (int r = 0; r < 16; ++r)
        red[((wave * NT + tm * TN + tn) * 16 + r) * 64 + lane] = PC ? __int_as_float(acc[tm][tn][r]) : y[tm][tn][r];
  __syncthreads();
  const int g = wave;
  float v[TM][TN][4];
#pragma unroll
  for (int tm = 0; tm < TM; ++tm)
#pragma unroll
    for (int tn = 0; tn < TN; ++tn)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int r = 4 * g + q, t = tm * TN + tn;
        if constexpr (PC) {  // int32 sums: exact in any order; raw bits while split
          int u = __float_as_int(red[(t * 16 + r) * 64 + lane]);
#pragma unroll
          for (int w = 1; w < 4; ++w) u += __float_as_int(red[((w * NT + t) * 16 + r) * 64 + lane]);
          v[tm][tn][q] = __int_as_float(u);
        } else {
          float u = red[(t * 16 + r) * 64 + lane];
#pragma unroll
          for (int w = 1; w < 4; ++w) u += red[((w * NT + t) * 16 + r) * 64 + lane];
          v[tm][tn][q] = u;
        }
      }

  if (S > 1) {
    // this K range's sums, [row][col] of the BM x BN block (rows < M)
    float* P = a.partial + (static_cast<size_t>(blockIdx.y * (N / BN) + strip) * S + range) * (BM * BN);
#pragma unroll
    for (int tm = 0; tm < TM; ++tm)
#pragma unroll
      for (int tn = 0; tn < TN; ++tn)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int row = tm * 32 + 8 * g + 4 * h + q;
          if (row < rows) P[row * BN + 32 * tn + col] = v[tm][tn][q];
        }
    return;
  }
  if constexpr (PC) {  // the one conversion, with the column's step (widened codes: factor 16)
#pragma unroll
    for (int tn = 0; tn < TN; ++tn) {
      const float wpc = f16_to_f32(a.w_scale[n0 + 32 * tn + col]) * 0.0625f;
#pragma unroll
      for (int tm = 0; tm < TM; ++tm)
#pragma unroll
        for (int q = 0; q < 4; ++q) v[tm][tn][q] = static_cast<float>(__float_as_int(v[tm][tn][q])) * wpc;
    }
  }
  // epilogue: row factor (8-bit: r_i; 4-bit: kappa_i = 1 / gamma_s(i), the
  // compensation of Eq. 8), fetched from the lane that loaded it; bias; cast.
  // A quad transpose gives each lane four consecutive channels of one row.
  constexpr bool kGelu = EPI == kEpiGelu;
  float rowf = 1.0f, bias[TN];
#pragma unroll
  for (int tn = 0; tn < TN; ++tn) bias[tn] = 0.0f;
  if constexpr (EPI == kEpiOut || kGelu) {
    const int m = m0 + min(lane, rows - 1);
    if constexpr (QX)
      rowf = qdelta / a.gamma[a.step * a.S + a.tok2stream[m]];  // r_i = Delta / gamma_s(i), as the first kernel
    else if constexpr (ABITS == 8)
      rowf = static_cast<const float*>(a.act_scale)[m];
    else
      rowf = 1.0f / a.gamma[a.step * a.S + a.tok2stream[m]];
    if (a.bias != nullptr) {
#pragma unroll
      for (int tn = 0; tn < TN; ++tn) bias[tn] = bf16_to_f32(a.bias[n0 + 32 * tn + col]);
    }
  }
  // GELU epilogue: the next layer's gain of the lane's row, its 1 / Delta,
  // and the D^-1 of the four columns each lane holds after the transpose;
  // 8-bit: the first strip's first wave writes the next layer's row scales
  float gain = 0.0f, ninv = 0.0f, ndinv[TN][4];
  uint32_t nstep16 = 0;  // 4-bit: the next layer's fp16 step
  if constexpr (kGelu) {
    const NextQuant& q = a.nq;
    gain = q.gamma[q.step * q.S + q.tok2stream[m0 + min(lane, rows - 1)]];
    float ndelta;
    if constexpr (ABITS == 8) {
      ndelta = q.clip[q.step] / 127.0f;
      ninv = 1.0f / ndelta;
      if (__builtin_isinf(ninv)) ninv = 0.0f;
    } else {
      nstep16 = static_step4(q.clip[q.step], ndelta, ninv);
    }
#pragma unroll
    for (int tn = 0; tn < TN; ++tn) {
      const float4 d = q.dinv != nullptr ? *reinterpret_cast<const float4*>(q.dinv + n0 + 32 * tn + (lane & 28))
                                         : make_float4(1.0f, 1.0f, 1.0f, 1.0f);
      ndinv[tn][0] = d.x;
      ndinv[tn][1] = d.y;
      ndinv[tn][2] = d.z;
      ndinv[tn][3] = d.w;
    }
    if constexpr (ABITS == 8) {
      if (n0 == 0 && g == 0 && lane < rows) q.r[m0 + lane] = ndelta / gain;
    }
  }
  const int rf_bits = __float_as_int(rowf);
  const bool f32out = EPI == kEpiPartial || a.out_dtype == SQ_OUT_F32;
#pragma unroll
  for (int t = 0; t < TM * TN; ++t) {
    const int tm = t / TN, tn = t % TN;
    float o[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const float rf = __int_as_float(__builtin_amdgcn_ds_bpermute((tm * 32 + 8 * g + 4 * h + q) * 4, rf_bits));
      o[q] = EPI == kEpiPartial ? v[tm][tn][q] : __builtin_fmaf(v[tm][tn][q], rf, bias[tn]);
    }
    quad_transpose(o, lane);
    const int row = tm * 32 + 8 * g + 4 * h + (lane & 3);
    const int n = n0 + 32 * tn + (lane & 28);
    float grow = 0.0f;
    if constexpr (kGelu) grow = __int_as_float(__builtin_amdgcn_ds_bpermute(row * 4, __float_as_int(gain)));
    if constexpr (kGelu && ABITS == 4) {
      // packed 4-bit codes: in a run of eight, codes 0-3 (this lane when
      // n % 8 == 0) fill the low nibbles of four bytes and codes 4-7 (lane ^ 4)
      // the high ones; one fp16 step per row and 64-group
      uint32_t bits[4], neg[4];
      gelu_codes4_a4(o, ndinv[tn], grow, ninv, bits, neg);
      uint32_t nib = 0;
#pragma unroll
      for (int j = 0; j < 4; ++j) nib |= (bits[j] & 0xFu) << (4 * j);
      const uint32_t other = static_cast<uint32_t>(__shfl_xor(static_cast<int>(nib), 4, 64));
      if (row < rows) {
        const size_t m = static_cast<size_t>(m0 + row);
        if ((lane & 4) == 0) {
          uint32_t w = 0;
#pragma unroll
          for (int j = 0; j < 4; ++j) w |= (((nib >> (4 * j)) & 0xFu) | (((other >> (4 * j)) & 0xFu) << 4)) << (8 * j);
          *reinterpret_cast<uint32_t*>(static_cast<uint8_t*>(a.out) + m * (N / 2) + n / 2) = w;
        }
        if ((n & 63) == 0) static_cast<uint16_t*>(a.nq.scale)[m * (N / 64) + n / 64] = static_cast<uint16_t>(nstep16);
      }
      continue;
    }
    if (row < rows) {
      const size_t m = static_cast<size_t>(m0 + row);
      if constexpr (kGelu) {
        *reinterpret_cast<uint32_t*>(static_cast<int8_t*>(a.out) + m * N + n) = gelu_codes4(o, ndinv[tn], grow, ninv);
      } else if (f32out) {
        *reinterpret_cast<float4*>(static_cast<float*>(a.out) + m * N + n) = make_float4(o[0], o[1], o[2], o[3]);
      } else {
        uint2 w;
        if (a.out_dtype == SQ_OUT_BF16) {
          const bf16x2 lo = __builtin_convertvector((float2v){o[0], o[1]}, bf16x2);
          const bf16x2 hi = __builtin_convertvector((float2v){o[2], o[3]}, bf16x2);
          w = make_uint2(__builtin_bit_cast(uint32_t, lo), __builtin_bit_cast(uint32_t, hi));
        } else {
          w = make_uint2(f32_to_f16(o[0]) | (f32_to_f16(o[1]) << 16), f32_to_f16(o[2]) | (f32_to_f16(o[3]) << 16));
        }
        *reinterpret_cast<uint2*>(static_cast<uint16_t*>(a.out) + m * N + n) = w;
      }
    }
  }
}

// Second kernel of a split skinny GEMM: adds the `split` partial sums of every
// output in range order (int32 sums with one step per channel, then the one
// conversion) and finishes it as the skinny epilogue does.  Four adjacent
// outputs per thread.
template <int ABITS, int EPI, bool PC, bool QX = false, int BM = SK_BM, int BN = SK_BN>
__global__ __launch_bounds__(256) void gemm_skinny_tail_kernel(GemmArgs a) {
  const int strips = a.N / BN;
  const int g = blockIdx.x * 256 + threadIdx.x;  // one thread per 4 outputs of a BM x BN block
  const int blk = g / (BM * BN / 4);
  const int e = (g % (BM * BN / 4)) * 4;
  const int row = e / BN, c = e % BN;
  const int mb = blk / strips, strip = blk % strips;
  const int m = mb * BM + row, n = strip * BN + c;
  if (mb * BM >= a.M || m >= a.M) return;
  const float* P = a.partial + static_cast<size_t>(blk) * a.split * (BM * BN) + row * BN + c;
  // the epilogue's inputs first, so that their loads overlap the partial sums'
  constexpr bool kOut = EPI == kEpiOut || EPI == kEpiGelu;
  float rowf = 1.0f, bias[4] = {0.0f, 0.0f, 0.0f, 0.0f}, wpc[4];
  if constexpr (kOut) {
    rowf = QX ? (a.clip[a.step] / 127.0f) / a.gamma[a.step * a.S + a.tok2stream[m]]
              : ABITS == 8 ? static_cast<const float*>(a.act_scale)[m]
                           : 1.0f / a.gamma[a.step * a.S + a.tok2stream[m]];
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
  if constexpr (EPI == kEpiGelu && ABITS == 4) {  // packed codes (pairs of threads fill bytes) and fp16 steps
    const NextQuant& q = a.nq;
    float ndelta, ninv;
    const uint32_t nstep16 = static_step4(q.clip[q.step], ndelta, ninv);
    const float gain = q.gamma[q.step * q.S + q.tok2stream[m]];
    const float4 d4 = q.dinv != nullptr ? *reinterpret_cast<const float4*>(q.dinv + n) : make_float4(1.0f, 1.0f, 1.0f, 1.0f);
    const float dv[4] = {d4.x, d4.y, d4.z, d4.w};
    uint32_t bits[4], neg[4];
    gelu_codes4_a4(y, dv, gain, ninv, bits, neg);
    uint32_t nib = 0;
#pragma unroll
    for (int j = 0; j < 4; ++j) nib |= (bits[j] & 0xFu) << (4 * j);
    // the thread with the run's codes 4-7 is the next one (n + 4: lane ^ 1), on the same row
    const uint32_t other = static_cast<uint32_t>(__shfl_xor(static_cast<int>(nib), 1, 64));
    if ((n & 7) == 0) {
      uint32_t w = 0;
#pragma unroll
      for (int j = 0; j < 4; ++j) w |= (((nib >> (4 * j)) & 0xFu) | (((other >> (4 * j)) & 0xFu) << 4)) << (8 * j);
      *reinterpret_cast<uint32_t*>(static_cast<uint8_t*>(a.out) + static_cast<size_t>(m) * (a.N / 2) + n / 2) = w;
    }
    if ((n & 63) == 0) static_cast<uint16_t*>(q.scale)[static_cast<size_t>(m) * (a.N / 64) + n / 64] =
        static_cast<uint16_t>(nstep16);
  } else if constexpr (EPI == kEpiGelu) {  // the next layer's codes (and, from the first column, its row scale)
    const NextQuant& q = a.nq;
    const float ndelta = q.clip[q.step] / 127.0f;
    float ninv = 1.0f / ndelta;
    if (__builtin_isinf(ninv)) ninv = 0.0f;
    const float gain = q.gamma[q.step * q.S + q.tok2stream[m]];
    const float4 d4 = q.dinv != nullptr ? *reinterpret_cast<const float4*>(q.dinv + n) : make_float4(1.0f, 1.0f, 1.0f, 1.0f);
    const float dv[4] = {d4.x, d4.y, d4.z, d4.w};
    *reinterpret_cast<uint32_t*>(static_cast<int8_t*>(a.out) + static_cast<size_t>(m) * a.N + n) =
        gelu_codes4(y, dv, gain, ninv);
    if (n == 0) q.r[m] = ndelta / gain;
  } else if (EPI == kEpiPartial || a.out_dtype == SQ_OUT_F32) {
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

// K ranges per strip: S workgroups share a strip when that shortens its
// waves' stage chains by more than the second kernel costs.  Measured on
// MI355X: a stage costs a wave about 0.65 us, the second kernel and its
// launch about 5 us, i.e. about 8 stages.  At most the workgroups that fit at
// once (by LDS), and at least four stages (one per wave) in every range.
template <int ABITS, int BM, int BN>
int split_t(int32_t M, int32_t N, int32_t K) {
  const int blocks = (N / BN) * ((M + BM - 1) / BM);
  const int nkt = K / KT;
  const int smax = std::max(1, std::min(device_cus() * Sk<ABITS, false, BM, BN>::WGS_PER_CU / blocks, nkt / 4));
  int best = 1;
  double best_cost = (nkt + 3) / 4;
  for (int S = 2; S <= smax; ++S) {
    const double cost = (nkt / S + 3) / 4 + 8.0;
    if (cost < best_cost) best = S, best_cost = cost;
  }
  return best;
}

// Block shape for a layer (QX: always 64 x 32).  Rows: 32 when 64-row blocks
// of 32 channels would give fewer workgroups than CUs (measured at 64 and 128
// tokens on the 2B linears, fused call, graph-replayed: out 12-18 % faster,
// down up to 14 %, qkv at 64 tokens within 3 %).  Channels: 64 when 64 x 32
// blocks would outnumber the CUs: the activations are then read once per 64
// channels and half as many workgroups remain (measured 7-23 % faster at 128
// tokens on the 2B qkv and up projections and on the 14B ones at 64 and 128
// tokens, with 8- and 4-bit codes; even where two 4-bit 64 x 32 blocks fit
// on a CU).
struct SkPlan {
  int bm, bn;
};
SkPlan skinny_plan(int32_t M, int32_t N, bool qx) {
  if (qx) return {SK_BM, SK_BN};
  const int w = (N / SK_BN) * ((M + SK_BM - 1) / SK_BM);
  if (w < device_cus()) return {32, SK_BN};
  if (w > device_cus()) return {SK_BM, 64};
  return {SK_BM, SK_BN};
}

template <int ABITS>
int split_for(const SkPlan& p, int32_t M, int32_t N, int32_t K) {
  if (p.bm == 32) return split_t<ABITS, 32, SK_BN>(M, N, K);
  return p.bn == 64 ? split_t<ABITS, SK_BM, 64>(M, N, K) : split_t<ABITS, SK_BM, SK_BN>(M, N, K);
}

int skinny_split(int act_bits, int32_t M, int32_t N, int32_t K, bool qx = false) {
  const SkPlan p = skinny_plan(M, N, qx);
  return act_bits == 8 ? split_for<8>(p, M, N, K) : split_for<4>(p, M, N, K);
}

size_t partial_bytes_for(int act_bits, int32_t M, int32_t N, int32_t K, bool qx) {
  const int S = skinny_split(act_bits, M, N, K, qx);
  if (S <= 1) return 0;
  const SkPlan p = skinny_plan(M, N, qx);
  return static_cast<size_t>(N / p.bn) * ((M + p.bm - 1) / p.bm) * S * (p.bm * p.bn) * sizeof(float);
}

template <int ABITS, int EPI, bool PC, bool QX, int BM, int BN>
hipError_t launch_bm(const GemmArgs& a0, hipStream_t s, float* partial, size_t partial_bytes) {
  GemmArgs a = a0;
  int S = skinny_split(ABITS, a.M, a.N, a.K, QX);
  if (S > 1 && (partial == nullptr || partial_bytes < partial_bytes_for(ABITS, a.M, a.N, a.K, QX))) S = 1;
  a.split = S;
  a.partial = S > 1 ? partial : nullptr;
  const int strips = a.N / BN, mblocks = (a.M + BM - 1) / BM;
  hipLaunchKernelGGL((gemm_skinny_kernel<ABITS, EPI, PC, QX, BM, BN>), dim3(strips * S, mblocks), dim3(256), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || S == 1) return e;
  const int threads = strips * mblocks * (BM * BN / 4);
  // with QX the second kernel computes r_i itself, as the first does
  hipLaunchKernelGGL((gemm_skinny_tail_kernel<ABITS, EPI, PC, QX, BM, BN>), dim3((threads + 255) / 256), dim3(256), 0, s,
                     a);
  return hipGetLastError();
}

template <int ABITS, int EPI, bool PC, bool QX = false>
hipError_t launch_t(const GemmArgs& a, hipStream_t s, float* partial, size_t partial_bytes) {
  if constexpr (!QX) {
    const SkPlan p = skinny_plan(a.M, a.N, false);
    if (p.bm == 32) return launch_bm<ABITS, EPI, PC, false, 32, SK_BN>(a, s, partial, partial_bytes);
    if (p.bn == 64) return launch_bm<ABITS, EPI, PC, false, SK_BM, 64>(a, s, partial, partial_bytes);
  }
  return launch_bm<ABITS, EPI, PC, QX, SK_BM, SK_BN>(a, s, partial, partial_bytes);
}

}  // namespace

size_t skinny_partial_bytes(int act_bits, int32_t M, int32_t N, int32_t K) {
  // the larger of the plans with and without in-kernel quantization (the
  // single-kernel linear takes 64-row blocks whatever the shape)
  const size_t b = partial_bytes_for(act_bits, M, N, K, false);
  return act_bits == 8 ? std::max(b, partial_bytes_for(8, M, N, K, true)) : b;
}

hipError_t launch_skinny_static1(const GemmArgs& a, hipStream_t s, float* partial, size_t partial_bytes) {
  return a.w_group != KT ? launch_t<8, kEpiOut, true, true>(a, s, partial, partial_bytes)
                         : launch_t<8, kEpiOut, false, true>(a, s, partial, partial_bytes);
}

hipError_t launch_skinny(int act_bits, int epi, const GemmArgs& a, hipStream_t s, float* partial,
                         size_t partial_bytes) {
  if (act_bits == 8) {
    const bool pc = a.w_group != KT;  // then w_group == K (skinny_applies)
    switch (epi) {
      case kEpiOut:
        return pc ? launch_t<8, kEpiOut, true>(a, s, partial, partial_bytes)
                  : launch_t<8, kEpiOut, false>(a, s, partial, partial_bytes);
      case kEpiPartial:
        return pc ? launch_t<8, kEpiPartial, true>(a, s, partial, partial_bytes)
                  : launch_t<8, kEpiPartial, false>(a, s, partial, partial_bytes);
      case kEpiGelu:
        return pc ? launch_t<8, kEpiGelu, true>(a, s, partial, partial_bytes)
                  : launch_t<8, kEpiGelu, false>(a, s, partial, partial_bytes);
    }
  } else {
    switch (epi) {
      case kEpiOut: return launch_t<4, kEpiOut, false>(a, s, partial, partial_bytes);
      case kEpiPartial: return launch_t<4, kEpiPartial, false>(a, s, partial, partial_bytes);
      case kEpiGelu: return launch_t<4, kEpiGelu, false>(a, s, partial, partial_bytes);
    }
  }
  return hipErrorInvalidValue;
}

}  // namespace sq
