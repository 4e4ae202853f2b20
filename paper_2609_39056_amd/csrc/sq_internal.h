// Internal declarations shared by the HIP translation units of libsq.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "sq.h"

namespace sq {

constexpr int kA4Group = 64;      // activation group of 4-bit codes along K
constexpr int kKTile = 128;       // K extent of one GEMM pipeline stage
constexpr int kMaxK = 32768;

// ---------------------------------------------------------------- number formats
__device__ __forceinline__ float bf16_to_f32(uint32_t bits16) {
  return __uint_as_float(bits16 << 16);
}

// fp32 -> bf16, round to nearest even (finite inputs).
__device__ __forceinline__ uint32_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return u >> 16;
}

// fp32 -> fp16 bits with the hardware conversion (round to nearest even).
__device__ __forceinline__ uint32_t f32_to_f16(float f) {
  _Float16 h = static_cast<_Float16>(f);
  return static_cast<uint32_t>(__builtin_bit_cast(uint16_t, h));
}

__device__ __forceinline__ float f16_to_f32(uint32_t bits16) {
  return static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(bits16)));
}

// Two's-complement nibbles of one packed dword (codes k0..k7 with k_b in the
// low and k_{b+4} in the high nibble of byte b) -> two dwords of int8 bytes
// holding 16 * code: lo = (16k0, 16k1, 16k2, 16k3), hi = (16k4, .., 16k7).
// Placing a nibble in the top half of a byte multiplies its signed value by 16
// without any sign extension.
__device__ __forceinline__ void unpack_int4x8_times16(uint32_t p, uint32_t& lo, uint32_t& hi) {
  lo = (p << 4) & 0xF0F0F0F0u;
  hi = p & 0xF0F0F0F0u;
}

// ---------------------------------------------------------------- launch grids
// A launch of n workgroups as an x * y grid with x <= 65536: a dispatch
// counts work-items per grid dimension in 32 bits, which one dimension of 256-
// thread workgroups would overflow from 2^24 workgroups on.  Kernels take
// flat_wg() as their index and leave when it is past n (the last grid row
// may be partly beyond).
inline dim3 wg_grid(size_t n) {
  const size_t x = n < 65536 ? (n == 0 ? 1 : n) : 65536;
  return dim3(static_cast<unsigned>(x), static_cast<unsigned>((n + x - 1) / x));
}
__device__ __forceinline__ size_t flat_wg() { return static_cast<size_t>(blockIdx.y) * gridDim.x + blockIdx.x; }

// ---------------------------------------------------------------- launch arguments
struct QuantArgs {
  const uint16_t* x;
  const int32_t* tok2stream;
  const float* gamma;
  const float* clip;
  const float* dinv;
  void* qx;
  void* scale;
  // 4-bit codes for the fp8 matrix cores (the fused linear's pipelined path):
  // when kc is set, qx holds one byte per code, the fp8 e4m3 value code * 2^-9
  // (sign and magnitude; |code| <= 7 is an exact subnormal), scale holds the
  // group steps sigma as fp32 (the fp16 value, widened) and kc holds the fp32
  // -8 * S * sigma * 2^-18 per (row, 64-group), S = the group's code sum.
  float* kc;
  int32_t M, K, S, step, range_mode;
};

enum EpiMode : int {
  kEpiOut = 0,      // full epilogue: row factor, bias, cast, store y
  kEpiPartial = 1,  // fp32 sum_b fp32(C^b) * s_b * Delta_W (no row factor / bias)
  kEpiInt32 = 2,    // int32 C (one block spanning K)
  kEpiDump = 3,     // int32 C^b of every block to acc_out[b][i][j]
  kEpiGelu = 4,     // row factor, bias, bf16, GELU, bf16, the next layer's STATIC codes to out
};

// The next linear's STATIC quantizer, applied by the kEpiGelu epilogue to
// GELU of this GEMM's bf16 output (codes to GemmArgs::out).  8-bit
// activations (this GEMM's and the next layer's): codes int8 [M][N], the row
// scales r = Delta / gamma_s(i) to `r`.  4-bit activations (both): Delta =
// fp16(clip / 7), and the codes in the form the next layer's GEMM takes:
// packed int4 [M][N/2] with fp16 steps [M][N/64] in `scale` (the
// weight-streaming GEMM, at most kSkinnyMaxM rows), or fp8 code bytes
// [M][N] with fp32 steps and kc = -8 S sigma 2^-18 per (row, 64-group) in
// `scale` and `kc` (the fp8 tiled GEMM).
struct NextQuant {
  const int32_t* tok2stream;
  const float* gamma;  // [num_steps][S]
  const float* dinv;   // D^-1 [N] or NULL
  const float* clip;   // [num_steps]: Delta = clip[step] / 127 (8-bit) or fp16(clip[step] / 7) (4-bit)
  int32_t S, step;
  float* r;            // [M] (8-bit)
  void* scale;         // 4-bit: fp16 [M][N/64] (packed codes) or fp32 [M][N/64] (fp8 code bytes)
  float* kc;           // 4-bit fp8 code bytes: [M][N/64]
};

struct GemmArgs {
  const void* qx;           // int8 [M][K] or packed int4 [M][K/2]
  const void* act_scale;    // fp32 r [M] (8-bit) or fp16 sigma [M][K/64] (4-bit); may be NULL in partial modes
  const int32_t* tok2stream;  // 4-bit kappa: s(i)
  const float* gamma;       // 4-bit kappa: gamma table
  int32_t S, step;
  const float* kc;          // 4-bit codes as fp8 bytes (see QuantArgs::kc); NULL: packed int4
  const uint8_t* qw;
  const uint16_t* w_scale;
  const uint16_t* bias;
  void* out;                // y, partial sums, int32 C or block dump
  int32_t M, N, K, w_group;
  int32_t out_dtype;
  // Split-K tail (set by launch_gemm): output tiles [0, ndp) of the logical
  // order are computed whole; each of the remaining ones is computed by
  // `split` workgroups over consecutive K ranges, which leave fp32 partial
  // sums in `partial`, and one more kernel adds them up and finishes the tile.
  int32_t ndp, split;
  float* partial;
  // the single-kernel linear (launch_skinny_static1): qx holds X (bf16 [M][K])
  // and the kernel quantizes it with STATIC thresholds, D^-1 and the gains
  const float* dinv;
  const float* clip;
  NextQuant nq;  // kEpiGelu only
};

// Bytes of the partial-sum buffer the split-K tail may use for a GEMM of this
// shape (0 when it never splits); any buffer at least this large lets
// launch_gemm choose its plan freely, a smaller one restricts it.
size_t gemm_partial_bytes(int act_bits, int32_t M, int32_t N, int32_t K, int32_t w_group);

// Compute units of the current device (256 when there is none), capped at 256.
int device_cus();

// Weight-streaming GEMM for M <= kSkinnyMaxM (epi kEpiOut, kEpiPartial, or
// kEpiGelu with 8-bit activations):
// 4-bit activations with any weight groups, 8-bit ones with 128-wide groups
// or one step per output channel.  Splits K across workgroups when `partial`
// holds skinny_partial_bytes(...) bytes.
constexpr int kSkinnyMaxM = 128;
inline bool skinny_applies(int act_bits, int32_t M, int32_t K, int32_t w_group) {
  return M <= kSkinnyMaxM && (act_bits == 4 || w_group == kKTile || w_group == K);
}
// 4-bit activations take the fp8 pipelined GEMM in the fused linear whenever
// the weight-streaming kernel does not apply (more than 128 tokens).
inline bool a4_fp8_path(int32_t M, int32_t K, int32_t w_group) { return !skinny_applies(4, M, K, w_group); }
size_t skinny_partial_bytes(int act_bits, int32_t M, int32_t N, int32_t K);
// The STATIC single-kernel W4A8 linear for few tokens (skinny_applies(8, ...)):
// the weight-streaming GEMM with the first kernel's quantization done on each
// stage in LDS; a.qx = X, a.dinv, a.clip, a.gamma, a.tok2stream, a.step, a.S
// set; EPI kEpiOut.  Splits K like launch_skinny (8-bit).
hipError_t launch_skinny_static1(const GemmArgs& a, hipStream_t s, float* partial, size_t partial_bytes);
hipError_t launch_skinny(int act_bits, int epi, const GemmArgs& a, hipStream_t s, float* partial,
                         size_t partial_bytes);

struct PackArgs {
  const float* w;
  const float* d;
  uint8_t* qw;
  uint16_t* w_scale;
  int32_t N, K, w_group;
};

// The fused linear (8- or 4-bit activations) with its workspace given: the
// same validation and kernels as sq_linear_w4a8 / sq_linear_w4a4.
sq_status linear_fused_on(int32_t bits, const uint16_t* x, int32_t M, const sq_act_params* act, const sq_weight* w,
                          void* y, int32_t out_dtype, void* ws, size_t ws_bytes, hipStream_t stream);

// ---------------------------------------------------------------- launchers (return hipError_t)
hipError_t launch_quantize_act(int act_bits, const QuantArgs& a, hipStream_t s);
hipError_t launch_pack_weights(const PackArgs& a, hipStream_t s);
// `partial` / `partial_bytes`: scratch for the split-K tail (may be NULL / 0:
// every tile is then computed whole).
hipError_t launch_gemm(int act_bits, int epi, const GemmArgs& a, hipStream_t s, float* partial = nullptr,
                       size_t partial_bytes = 0);
// The 8-bit GEMM with the kEpiGelu epilogue (a.nq set, a.out the codes): the
// pipelined kernel with 128-wide weight groups (more than kSkinnyMaxM rows),
// or the weight-streaming one (128-wide groups or one step per channel).
hipError_t launch_gemm_gelu_quant(const GemmArgs& a, hipStream_t s, float* partial, size_t partial_bytes);
// The same for 4-bit activations (this GEMM's and the next layer's): the
// weight-streaming GEMM on packed codes (at most kSkinnyMaxM rows; next
// layer's codes packed, fp16 steps) or the fp8 tiled GEMM (a.kc set; next
// layer's codes as fp8 bytes, fp32 steps and kc).
hipError_t launch_gemm_gelu_quant4(const GemmArgs& a, hipStream_t s, float* partial, size_t partial_bytes);
// GELU of n bf16 values to bf16 (the fp32 sequence of gelu.h).
hipError_t launch_gelu_bf16(const uint16_t* x, size_t n, uint16_t* y, hipStream_t s);

// unfused stages
struct UnfusedArgs {
  const uint16_t* x;
  const int32_t* tok2stream;
  const float* gamma;
  const float* clip;
  const float* dinv;
  const uint8_t* qw;
  const uint16_t* w_scale;
  const uint16_t* bias;
  int32_t M, K, N, S, step, range_mode, act_bits, w_group, out_dtype;
  // workspace views
  float* xt;        // [M][K] X D^-1
  float* gmax;      // [M][groups] amax of X D^-1
  float* xh;        // [M][K] X D^-1 gamma
  void* qx;         // codes
  void* qscale;     // 8-bit: fp32 Delta [M]; 4-bit: fp16 sigma [M][K/64]
  void* gemm_out;   // fp32 partial [M][N] or int32 C [M][N]
  float* y1;        // [M][N] after the activation step
  float* y2;        // [M][N] after the inverse-gain compensation
  void* y;          // final output
};
hipError_t launch_unfused(const UnfusedArgs& a, hipStream_t s);

// calibration objective (Sec. 4.3, Eq. 9)
constexpr int32_t kCalibMaxStreams = 4096;  // streams of one objective (an LDS histogram)
struct CalibRefArgs {
  const uint16_t* x;
  const float* dinv;
  const uint8_t* qw;
  const uint16_t* w_scale;
  const float* wf;  // fp32 W [N][K]: the target is X W (no D^-1, no codes); NULL: X~ W^ from qw / w_scale
  double* y;        // [M][N]
  int32_t M, N, K, w_group;
};
// per-channel amax of |x| (bf16 [M][K]) and |w| (fp32 [N][K]) as fp32 bits
hipError_t launch_channel_amax(const uint16_t* x, int32_t M, const float* w, int32_t N, int32_t K,
                               uint32_t* ax_bits, uint32_t* aw_bits, hipStream_t s);
// d = clamp(ax^alpha / aw^(1 - alpha), 2^-6, 2^6) (fp64, 1 where an amax is 0), dinv = 1 / d
hipError_t launch_smooth_scales(const uint32_t* ax_bits, const uint32_t* aw_bits, int32_t K, float alpha, float* d,
                                float* dinv, hipStream_t s);
hipError_t launch_fill_f32(float* p, int32_t n, float v, hipStream_t s);
hipError_t launch_calib_reference(const CalibRefArgs& a, hipStream_t s);
// counts[s] = tokens of stream s (ids outside [0, S) are not counted)
hipError_t launch_calib_counts(const int32_t* tok2stream, int32_t M, int32_t S, int32_t* counts, hipStream_t s);
// err[i] = omega_s(i) / n_s(i) * ||y_i - ref_i||^2, then *out = sum_i err[i]
hipError_t launch_calib_error(const float* yq, const double* ref, const int32_t* tok2stream,
                              const int32_t* counts, const double* omega, int32_t M, int32_t N, int32_t S,
                              double* err, double* out, hipStream_t s);

// constrained compass search for Eq. 9 (at most kCalibSearchMaxStreams
// streams: one thread per candidate, 2 (S + 1) of them)
constexpr int32_t kCalibSearchMaxStreams = 64;
struct SearchBounds {
  float gamma_min, gamma_max, clip_min, clip_max, clip_init, log_step;
};
hipError_t launch_calib_search_init(const SearchBounds& b, int32_t S, double* st, double* u, float* gamma,
                                    float* clip, hipStream_t s);
hipError_t launch_calib_propose(const SearchBounds& b, int32_t S, const int32_t* counts, const double* st,
                                const double* u, double* cand_u, double* cand_v, float* cand_gamma,
                                float* cand_clip, hipStream_t s);
hipError_t launch_calib_select(int32_t S, const double* cand_obj, const double* cand_u, const double* cand_v,
                               const float* cand_gamma, const float* cand_clip, double* st, double* u,
                               float* gamma, float* clip, double* objective, hipStream_t s);

// matrix-core rate probe (measurement hook)
int mfma_probe_workgroups();
hipError_t launch_mfma_probe(int32_t* sink, int32_t shape, int32_t iters, int32_t random, int32_t fold, hipStream_t s);
hipError_t launch_mfma_probe_f8f6(int32_t* sink, int32_t fmt, int32_t iters, int32_t random, int32_t fold,
                                  hipStream_t s);

}  // namespace sq
