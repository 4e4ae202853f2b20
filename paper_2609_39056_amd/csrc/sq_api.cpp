// Host side of the C ABI declared in sq.h: argument validation, workspace
// layout and kernel dispatch.  Nothing here allocates, frees or synchronizes.
#include <stdint.h>

#include <algorithm>
#include <cmath>

#include "sq_internal.h"

using namespace sq;

namespace {

constexpr int32_t kMaxM = 1 << 24;
constexpr int32_t kMaxN = 1 << 20;
constexpr size_t kAlign = 256;

size_t round_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

sq_status hip_status(hipError_t e) { return e == hipSuccess ? SQ_OK : SQ_ERR_HIP; }

bool valid_m(int32_t M) { return M >= 1 && M <= kMaxM; }
bool valid_k(int32_t K) { return K >= kKTile && K <= kMaxK && K % kKTile == 0; }
bool valid_n(int32_t N) { return N >= 64 && N <= kMaxN && N % 64 == 0; }

sq_status check_act(const sq_act_params* act, int32_t K) {
  if (act == nullptr || act->tok2stream == nullptr || act->gamma == nullptr) return SQ_ERR_NULL;
  if (act->act_bits != 8 && act->act_bits != 4) return SQ_ERR_UNSUPPORTED;
  if (act->range_mode != SQ_RANGE_DYNAMIC && act->range_mode != SQ_RANGE_STATIC) return SQ_ERR_UNSUPPORTED;
  if (act->range_mode == SQ_RANGE_STATIC && act->clip == nullptr) return SQ_ERR_NULL;
  if (act->num_streams < 1 || act->num_steps < 1) return SQ_ERR_SHAPE;
  if (act->step < 0 || act->step >= act->num_steps) return SQ_ERR_SHAPE;
  if (!valid_k(K)) return SQ_ERR_SHAPE;
  if (!aligned(act->tok2stream, 4) || !aligned(act->gamma, 4)) return SQ_ERR_ALIGN;
  if (act->clip != nullptr && !aligned(act->clip, 4)) return SQ_ERR_ALIGN;
  if (act->dinv != nullptr && !aligned(act->dinv, 16)) return SQ_ERR_ALIGN;
  return SQ_OK;
}

sq_status check_weight(const sq_weight* w) {
  if (w == nullptr || w->qw == nullptr || w->w_scale == nullptr) return SQ_ERR_NULL;
  if (!valid_k(w->K) || !valid_n(w->N)) return SQ_ERR_SHAPE;
  if (w->w_group < kKTile || w->w_group % kKTile != 0 || w->K % w->w_group != 0) return SQ_ERR_UNSUPPORTED;
  if (!aligned(w->qw, 16) || !aligned(w->w_scale, 4)) return SQ_ERR_ALIGN;
  if (w->bias != nullptr && !aligned(w->bias, 2)) return SQ_ERR_ALIGN;
  return SQ_OK;
}

bool valid_out(int32_t d) { return d == SQ_OUT_F32 || d == SQ_OUT_BF16 || d == SQ_OUT_F16; }

size_t qx_bytes(int32_t M, int32_t K, int32_t bits) {
  return bits == 8 ? static_cast<size_t>(M) * K : static_cast<size_t>(M) * K / 2;
}
size_t act_scale_bytes(int32_t M, int32_t K, int32_t bits) {
  return bits == 8 ? static_cast<size_t>(M) * 4 : static_cast<size_t>(M) * (K / kA4Group) * 2;
}

// Split-K partial sums of the GEMM: the larger of the plans for 128-wide
// weight groups and for one step per output channel (the cases that split),
// an upper bound for every w_group.
size_t gemm_ws_bytes(int32_t M, int32_t K, int32_t N, int32_t bits) {
  const size_t p = std::max(gemm_partial_bytes(bits, M, N, K, kKTile), gemm_partial_bytes(bits, M, N, K, K));
  return std::max<size_t>(kAlign, round_up(p));
}

// fused workspace: Q_X | scales | (fp8 4-bit codes: kc) | GEMM partial sums,
// each 256-byte aligned.  With 4-bit activations on the pipelined path
// (a4_fp8_path) Q_X holds one fp8 byte per code, the steps are fp32 and kc
// follows them.
struct FusedWs {
  void* qx;
  void* scale;
  float* kc;
  float* partial;
  size_t partial_bytes;
};
size_t kc_bytes(int32_t M, int32_t K) { return static_cast<size_t>(M) * (K / kA4Group) * 4; }
FusedWs fused_ws(void* ws, size_t ws_bytes, int32_t M, int32_t K, int32_t bits, bool f8) {
  uint8_t* p = static_cast<uint8_t*>(ws);
  FusedWs f;
  const size_t q = round_up(f8 ? static_cast<size_t>(M) * K : qx_bytes(M, K, bits));
  f.qx = p;
  f.scale = p + q;
  size_t off = q + round_up(f8 ? kc_bytes(M, K) : act_scale_bytes(M, K, bits));  // fp8 codes: fp32 steps
  f.kc = nullptr;
  if (f8) {
    f.kc = reinterpret_cast<float*>(p + off);
    off += round_up(kc_bytes(M, K));
  }
  f.partial = reinterpret_cast<float*>(p + off);
  f.partial_bytes = ws_bytes - off;
  return f;
}

// Sized for the larger layout (fp8 codes and kc for 4-bit activations): the
// weight's group width, which picks the path, is not an argument here.
size_t fused_ws_bytes(int32_t M, int32_t K, int32_t N, int32_t bits) {
  if (bits == 4)  // fp8 codes [M][K], fp32 steps and kc [M][K/64] each
    return round_up(static_cast<size_t>(M) * K) + 2 * round_up(kc_bytes(M, K)) + gemm_ws_bytes(M, K, N, bits);
  return round_up(qx_bytes(M, K, bits)) + round_up(act_scale_bytes(M, K, bits)) + gemm_ws_bytes(M, K, N, bits);
}

// calibration workspace: the fused linear's | y of one candidate fp32 [M][N] |
// per-row errors fp64 [M] | stream counts int32 [S]
constexpr int32_t kCalibMaxCandidates = 1 << 16;
constexpr int32_t kCalibSearchMaxRounds = 1024;
size_t calib_ws_bytes(int32_t M, int32_t K, int32_t N, int32_t bits, int32_t S) {
  return fused_ws_bytes(M, K, N, bits) + round_up(static_cast<size_t>(M) * N * 4) +
         round_up(static_cast<size_t>(M) * 8) + round_up(static_cast<size_t>(S) * 4);
}

// search state after the calibration workspace: st fp64 [4] | u fp64 [S] |
// candidates' log gains fp64 [C][S] | log thresholds fp64 [C] | objectives
// fp64 [C] | gains fp32 [C][S] | thresholds fp32 [C], C = 2 (S + 1)
struct SearchWs {
  double *st, *u, *cand_u, *cand_v, *cand_obj;
  float *cand_gamma, *cand_clip;
};
size_t search_extra_bytes(int32_t S, SearchWs* out = nullptr, uint8_t* base = nullptr) {
  const size_t C = 2 * (static_cast<size_t>(S) + 1);
  const size_t parts[7] = {4 * 8, S * 8ull, C * S * 8, C * 8, C * 8, C * S * 4, C * 4};
  size_t off = 0;
  void* ptr[7];
  for (int i = 0; i < 7; ++i) {
    ptr[i] = base + off;
    off += round_up(parts[i]);
  }
  if (out != nullptr) {
    out->st = static_cast<double*>(ptr[0]);
    out->u = static_cast<double*>(ptr[1]);
    out->cand_u = static_cast<double*>(ptr[2]);
    out->cand_v = static_cast<double*>(ptr[3]);
    out->cand_obj = static_cast<double*>(ptr[4]);
    out->cand_gamma = static_cast<float*>(ptr[5]);
    out->cand_clip = static_cast<float*>(ptr[6]);
  }
  return off;
}

// scaling-objective area after the calibration workspace: amax bits of X and
// W [K] | d [K] | dinv [K] | packed Q(D W) [N][K/2] | fp16 steps [K/w_group][N]
// | a one-step gain table of ones [R]
struct ScalingWs {
  uint32_t *ax, *aw;
  float *d, *dinv, *ones;
  uint8_t* qw;
  uint16_t* w_scale;
};
size_t scaling_extra_bytes(int32_t K, int32_t N, int32_t w_group, int32_t R, ScalingWs* out = nullptr,
                           uint8_t* base = nullptr) {
  const size_t parts[7] = {4ull * K, 4ull * K, 4ull * K, 4ull * K, static_cast<size_t>(N) * K / 2,
                           static_cast<size_t>(K / w_group) * N * 2, 4ull * R};
  size_t off = 0;
  void* ptr[7];
  for (int i = 0; i < 7; ++i) {
    ptr[i] = base + off;
    off += round_up(parts[i]);
  }
  if (out != nullptr) {
    out->ax = static_cast<uint32_t*>(ptr[0]);
    out->aw = static_cast<uint32_t*>(ptr[1]);
    out->d = static_cast<float*>(ptr[2]);
    out->dinv = static_cast<float*>(ptr[3]);
    out->qw = static_cast<uint8_t*>(ptr[4]);
    out->w_scale = static_cast<uint16_t*>(ptr[5]);
    out->ones = static_cast<float*>(ptr[6]);
  }
  return off;
}

size_t unfused_ws_bytes(int32_t M, int32_t K, int32_t N, int32_t bits) {
  const size_t mk4 = round_up(static_cast<size_t>(M) * K * 4);
  const size_t mn4 = round_up(static_cast<size_t>(M) * N * 4);
  const size_t groups = bits == 8 ? 1 : K / kA4Group;
  return 2 * mk4 + round_up(static_cast<size_t>(M) * groups * 4) + round_up(qx_bytes(M, K, bits)) +
         round_up(act_scale_bytes(M, K, bits)) + 3 * mn4;
}

sq_status quantize(const uint16_t* x, int32_t M, int32_t K, const sq_act_params* act, void* qx,
                   void* scale, hipStream_t stream, float* kc = nullptr) {
  QuantArgs q;
  q.kc = kc;
  q.x = x;
  q.tok2stream = act->tok2stream;
  q.gamma = act->gamma;
  q.clip = act->clip;
  q.dinv = act->dinv;
  q.qx = qx;
  q.scale = scale;
  q.M = M;
  q.K = K;
  q.S = act->num_streams;
  q.step = act->step;
  q.range_mode = act->range_mode;
  return hip_status(launch_quantize_act(act->act_bits, q, stream));
}

GemmArgs gemm_args(const void* qx, const void* scale, int32_t M, const sq_act_params* act,
                   const sq_weight* w, void* out, int32_t out_dtype) {
  GemmArgs g{};
  g.qx = qx;
  g.act_scale = scale;
  if (act != nullptr) {
    g.tok2stream = act->tok2stream;
    g.gamma = act->gamma;
    g.S = act->num_streams;
    g.step = act->step;
  }
  g.qw = w->qw;
  g.w_scale = w->w_scale;
  g.bias = w->bias;
  g.out = out;
  g.M = M;
  g.N = w->N;
  g.K = w->K;
  g.w_group = w->w_group;
  g.out_dtype = out_dtype;
  return g;
}

sq_status linear_fused(int32_t bits, const uint16_t* x, int32_t M, const sq_act_params* act,
                       const sq_weight* w, void* y, int32_t out_dtype, void* ws, size_t ws_bytes,
                       hipStream_t stream) {
  if (x == nullptr || y == nullptr || ws == nullptr) return SQ_ERR_NULL;
  sq_status st = check_weight(w);
  if (st != SQ_OK) return st;
  st = check_act(act, w->K);
  if (st != SQ_OK) return st;
  if (act->act_bits != bits) return SQ_ERR_UNSUPPORTED;
  if (!valid_m(M)) return SQ_ERR_SHAPE;
  if (!valid_out(out_dtype)) return SQ_ERR_UNSUPPORTED;
  if (!aligned(x, 16) || !aligned(y, 16) || !aligned(ws, 16)) return SQ_ERR_ALIGN;
  if (ws_bytes < fused_ws_bytes(M, w->K, w->N, bits)) return SQ_ERR_WORKSPACE;
  const bool f8 = bits == 4 && a4_fp8_path(M, w->K, w->w_group);
  FusedWs f = fused_ws(ws, ws_bytes, M, w->K, bits, f8);
  st = quantize(x, M, w->K, act, f.qx, f.scale, stream, f.kc);
  if (st != SQ_OK) return st;
  GemmArgs g = gemm_args(f.qx, f.scale, M, act, w, y, out_dtype);
  g.kc = f.kc;
  return hip_status(launch_gemm(bits, kEpiOut, g, stream, f.partial, f.partial_bytes));
}

}  // namespace

// The fused linear on a caller-chosen workspace (the library's static scratch
// for the allocation-free entry point).
sq_status sq::linear_fused_on(int32_t bits, const uint16_t* x, int32_t M, const sq_act_params* act,
                              const sq_weight* w, void* y, int32_t out_dtype, void* ws, size_t ws_bytes,
                              hipStream_t stream) {
  return linear_fused(bits, x, M, act, w, y, out_dtype, ws, ws_bytes, stream);
}

namespace {

// One candidate of Eq. 9: the fused linear in STATIC mode with one-step
// tables (gamma [S], clip [1], both device pointers) and no bias into fp32,
// then the weighted squared error against y_ref into *out.
struct CalibEval {
  const uint16_t* x;
  int32_t M, S, act_bits;
  const int32_t* tok2stream;
  const float* dinv;
  sq_weight wt;
  const double* y_ref;
  const double* omega;
  void* fused_ws;
  size_t fused_bytes;
  float* yq;
  double* err;
  int32_t* counts;
};

CalibEval calib_eval_setup(const uint16_t* x, int32_t M, const int32_t* tok2stream, int32_t S, const float* dinv,
                           int32_t act_bits, const sq_weight* w, const double* y_ref, const double* omega,
                           void* workspace) {
  CalibEval e;
  e.x = x;
  e.M = M;
  e.S = S;
  e.act_bits = act_bits;
  e.tok2stream = tok2stream;
  e.dinv = dinv;
  e.wt = *w;
  e.wt.bias = nullptr;  // the bias is on both sides of Eq. 9 and cancels
  e.y_ref = y_ref;
  e.omega = omega;
  uint8_t* p = static_cast<uint8_t*>(workspace);
  e.fused_ws = p;
  e.fused_bytes = fused_ws_bytes(M, w->K, w->N, act_bits);
  e.yq = reinterpret_cast<float*>(p + e.fused_bytes);
  e.err = reinterpret_cast<double*>(p + e.fused_bytes + round_up(static_cast<size_t>(M) * w->N * 4));
  e.counts = reinterpret_cast<int32_t*>(reinterpret_cast<uint8_t*>(e.err) + round_up(static_cast<size_t>(M) * 8));
  return e;
}

sq_status calib_eval_range(const CalibEval& e, const float* gamma, const float* clip, int32_t range_mode, double* out,
                           hipStream_t stream) {
  sq_act_params a{};
  a.tok2stream = e.tok2stream;
  a.gamma = gamma;
  a.clip = clip;
  a.dinv = e.dinv;
  a.num_streams = e.S;
  a.num_steps = 1;
  a.step = 0;
  a.range_mode = range_mode;
  a.act_bits = e.act_bits;
  sq_status st = linear_fused(e.act_bits, e.x, e.M, &a, &e.wt, e.yq, SQ_OUT_F32, e.fused_ws, e.fused_bytes, stream);
  if (st != SQ_OK) return st;
  return hip_status(launch_calib_error(e.yq, e.y_ref, e.tok2stream, e.counts, e.omega, e.M, e.wt.N, e.S, e.err,
                                       out, stream));
}

sq_status calib_eval(const CalibEval& e, const float* gamma, const float* clip, double* out, hipStream_t stream) {
  return calib_eval_range(e, gamma, clip, SQ_RANGE_STATIC, out, stream);
}

}  // namespace

extern "C" {

const char* sq_status_string(int32_t status) {
  switch (status) {
    case SQ_OK: return "SQ_OK";
    case SQ_ERR_NULL: return "SQ_ERR_NULL: a required pointer is NULL";
    case SQ_ERR_SHAPE: return "SQ_ERR_SHAPE: a size, step index or stream count is out of range";
    case SQ_ERR_ALIGN: return "SQ_ERR_ALIGN: a pointer is not aligned as required";
    case SQ_ERR_UNSUPPORTED: return "SQ_ERR_UNSUPPORTED: bits, group size, range mode or dtype not supported";
    case SQ_ERR_WORKSPACE: return "SQ_ERR_WORKSPACE: workspace too small";
    case SQ_ERR_HIP: return "SQ_ERR_HIP: a kernel launch failed";
    default: return "unknown sq_status";
  }
}

size_t sq_workspace_bytes(int32_t variant, int32_t M, int32_t K, int32_t N, int32_t act_bits) {
  if (!valid_m(M) || !valid_k(K) || !valid_n(N) || (act_bits != 8 && act_bits != 4)) return 0;
  if (variant == SQ_VARIANT_FUSED) return fused_ws_bytes(M, K, N, act_bits);
  if (variant == SQ_VARIANT_UNFUSED) return unfused_ws_bytes(M, K, N, act_bits);
  if (variant == SQ_VARIANT_GEMM) return gemm_ws_bytes(M, K, N, act_bits);
  return 0;
}

sq_status sq_pack_weights(const float* w, const float* d, int32_t N, int32_t K, int32_t w_group,
                          uint8_t* qw, uint16_t* w_scale, hipStream_t stream) {
  if (w == nullptr || qw == nullptr || w_scale == nullptr) return SQ_ERR_NULL;
  if (!valid_k(K) || !valid_n(N)) return SQ_ERR_SHAPE;
  if (w_group < kKTile || w_group % kKTile != 0 || K % w_group != 0) return SQ_ERR_UNSUPPORTED;
  if (!aligned(w, 16) || !aligned(qw, 16) || !aligned(w_scale, 4)) return SQ_ERR_ALIGN;
  if (d != nullptr && !aligned(d, 16)) return SQ_ERR_ALIGN;
  PackArgs p{w, d, qw, w_scale, N, K, w_group};
  return hip_status(launch_pack_weights(p, stream));
}

sq_status sq_quantize_act(const uint16_t* x, int32_t M, int32_t K, const sq_act_params* act,
                          void* qx, void* act_scale, hipStream_t stream) {
  if (x == nullptr || qx == nullptr || act_scale == nullptr) return SQ_ERR_NULL;
  sq_status st = check_act(act, K);
  if (st != SQ_OK) return st;
  if (!valid_m(M)) return SQ_ERR_SHAPE;
  if (!aligned(x, 16) || !aligned(qx, 16)) return SQ_ERR_ALIGN;
  if (!aligned(act_scale, 4)) return SQ_ERR_ALIGN;
  return quantize(x, M, K, act, qx, act_scale, stream);
}

sq_status sq_gemm_w4a8(const int8_t* qx, const float* row_scale, int32_t M, const sq_weight* w,
                       void* y, int32_t out_dtype, void* workspace, size_t ws_bytes, hipStream_t stream) {
  if (qx == nullptr || row_scale == nullptr || y == nullptr) return SQ_ERR_NULL;
  sq_status st = check_weight(w);
  if (st != SQ_OK) return st;
  if (!valid_m(M)) return SQ_ERR_SHAPE;
  if (!valid_out(out_dtype)) return SQ_ERR_UNSUPPORTED;
  if (!aligned(qx, 16) || !aligned(y, 16) || !aligned(row_scale, 4)) return SQ_ERR_ALIGN;
  if (workspace != nullptr && !aligned(workspace, 16)) return SQ_ERR_ALIGN;
  return hip_status(launch_gemm(8, kEpiOut, gemm_args(qx, row_scale, M, nullptr, w, y, out_dtype), stream,
                                static_cast<float*>(workspace), workspace ? ws_bytes : 0));
}

sq_status sq_gemm_w4a4(const uint8_t* qx, const uint16_t* group_scale, int32_t M,
                       const sq_act_params* act, const sq_weight* w, void* y, int32_t out_dtype,
                       void* workspace, size_t ws_bytes, hipStream_t stream) {
  if (qx == nullptr || group_scale == nullptr || y == nullptr) return SQ_ERR_NULL;
  sq_status st = check_weight(w);
  if (st != SQ_OK) return st;
  st = check_act(act, w->K);
  if (st != SQ_OK) return st;
  if (act->act_bits != 4) return SQ_ERR_UNSUPPORTED;
  if (!valid_m(M)) return SQ_ERR_SHAPE;
  if (!valid_out(out_dtype)) return SQ_ERR_UNSUPPORTED;
  if (!aligned(qx, 16) || !aligned(y, 16) || !aligned(group_scale, 4)) return SQ_ERR_ALIGN;
  if (workspace != nullptr && !aligned(workspace, 16)) return SQ_ERR_ALIGN;
  return hip_status(launch_gemm(4, kEpiOut, gemm_args(qx, group_scale, M, act, w, y, out_dtype), stream,
                                static_cast<float*>(workspace), workspace ? ws_bytes : 0));
}

sq_status sq_linear_w4a8(const uint16_t* x, int32_t M, const sq_act_params* act, const sq_weight* w,
                         void* y, int32_t out_dtype, void* workspace, size_t ws_bytes,
                         hipStream_t stream) {
  return linear_fused(8, x, M, act, w, y, out_dtype, workspace, ws_bytes, stream);
}

sq_status sq_linear_w4a4(const uint16_t* x, int32_t M, const sq_act_params* act, const sq_weight* w,
                         void* y, int32_t out_dtype, void* workspace, size_t ws_bytes,
                         hipStream_t stream) {
  return linear_fused(4, x, M, act, w, y, out_dtype, workspace, ws_bytes, stream);
}

sq_status sq_linear_w4a8_static1(const uint16_t* x, int32_t M, const sq_act_params* act, const sq_weight* w,
                                 void* y, int32_t out_dtype, void* workspace, size_t ws_bytes, hipStream_t stream) {
  if (x == nullptr || y == nullptr) return SQ_ERR_NULL;
  sq_status st = check_weight(w);
  if (st != SQ_OK) return st;
  st = check_act(act, w->K);
  if (st != SQ_OK) return st;
  if (act->act_bits != 8 || act->range_mode != SQ_RANGE_STATIC) return SQ_ERR_UNSUPPORTED;
  if (!valid_m(M)) return SQ_ERR_SHAPE;
  if (!skinny_applies(8, M, w->K, w->w_group)) return SQ_ERR_UNSUPPORTED;
  if (!valid_out(out_dtype)) return SQ_ERR_UNSUPPORTED;
  if (!aligned(x, 16) || !aligned(y, 16)) return SQ_ERR_ALIGN;
  if (workspace != nullptr && !aligned(workspace, 16)) return SQ_ERR_ALIGN;
  GemmArgs g = gemm_args(x, nullptr, M, act, w, y, out_dtype);
  g.dinv = act->dinv;
  g.clip = act->clip;
  return hip_status(launch_skinny_static1(g, stream, static_cast<float*>(workspace), workspace ? ws_bytes : 0));
}

sq_status sq_linear_w4a8_gelu_quant(const uint16_t* x, int32_t M, const sq_act_params* act, const sq_weight* w,
                                    const sq_act_params* act_next, int8_t* qx_next, float* r_next, void* workspace,
                                    size_t ws_bytes, hipStream_t stream) {
  if (x == nullptr || qx_next == nullptr || r_next == nullptr || workspace == nullptr) return SQ_ERR_NULL;
  sq_status st = check_weight(w);
  if (st != SQ_OK) return st;
  st = check_act(act, w->K);
  if (st != SQ_OK) return st;
  st = check_act(act_next, w->N);  // the next layer's input channels are this layer's outputs
  if (st != SQ_OK) return st;
  if (act->act_bits != 8 || act_next->act_bits != 8 || act_next->range_mode != SQ_RANGE_STATIC)
    return SQ_ERR_UNSUPPORTED;
  if (!valid_m(M)) return SQ_ERR_SHAPE;
  // 128-wide weight groups or one step per output channel (the weight-streaming
  // GEMM for few tokens, else the tiled ones)
  if (w->w_group != kKTile && w->w_group != w->K) return SQ_ERR_UNSUPPORTED;
  if (!aligned(x, 16) || !aligned(workspace, 16) || !aligned(qx_next, 4) || !aligned(r_next, 4)) return SQ_ERR_ALIGN;
  if (ws_bytes < fused_ws_bytes(M, w->K, w->N, 8)) return SQ_ERR_WORKSPACE;
  FusedWs f = fused_ws(workspace, ws_bytes, M, w->K, 8, false);
  st = quantize(x, M, w->K, act, f.qx, f.scale, stream);
  if (st != SQ_OK) return st;
  GemmArgs g = gemm_args(f.qx, f.scale, M, act, w, qx_next, SQ_OUT_BF16);
  g.nq.tok2stream = act_next->tok2stream;
  g.nq.gamma = act_next->gamma;
  g.nq.dinv = act_next->dinv;
  g.nq.clip = act_next->clip;
  g.nq.S = act_next->num_streams;
  g.nq.step = act_next->step;
  g.nq.r = r_next;
  return hip_status(launch_gemm_gelu_quant(g, stream, f.partial, f.partial_bytes));
}

sq_status sq_linear_w4a4_gelu_quant(const uint16_t* x, int32_t M, const sq_act_params* act, const sq_weight* w,
                                    const sq_act_params* act_next, void* qx_next, void* scale_next, float* kc_next,
                                    void* workspace, size_t ws_bytes, hipStream_t stream) {
  if (x == nullptr || qx_next == nullptr || scale_next == nullptr || workspace == nullptr) return SQ_ERR_NULL;
  sq_status st = check_weight(w);
  if (st != SQ_OK) return st;
  st = check_act(act, w->K);
  if (st != SQ_OK) return st;
  st = check_act(act_next, w->N);  // the next layer's input channels are this layer's outputs
  if (st != SQ_OK) return st;
  if (act->act_bits != 4 || act_next->act_bits != 4 || act_next->range_mode != SQ_RANGE_STATIC)
    return SQ_ERR_UNSUPPORTED;
  if (!valid_m(M)) return SQ_ERR_SHAPE;
  // more than 128 tokens: the fp8 tiled GEMM, and the next layer's codes in its form
  const bool f8 = a4_fp8_path(M, w->K, w->w_group);
  if (f8 && kc_next == nullptr) return SQ_ERR_NULL;
  if (!aligned(x, 16) || !aligned(workspace, 16) || !aligned(qx_next, 4) || !aligned(scale_next, f8 ? 4 : 2) ||
      (f8 && !aligned(kc_next, 4)))
    return SQ_ERR_ALIGN;
  if (ws_bytes < fused_ws_bytes(M, w->K, w->N, 4)) return SQ_ERR_WORKSPACE;
  FusedWs f = fused_ws(workspace, ws_bytes, M, w->K, 4, f8);
  st = quantize(x, M, w->K, act, f.qx, f.scale, stream, f.kc);
  if (st != SQ_OK) return st;
  GemmArgs g = gemm_args(f.qx, f.scale, M, act, w, qx_next, SQ_OUT_BF16);
  g.kc = f.kc;
  g.nq.tok2stream = act_next->tok2stream;
  g.nq.gamma = act_next->gamma;
  g.nq.dinv = act_next->dinv;
  g.nq.clip = act_next->clip;
  g.nq.S = act_next->num_streams;
  g.nq.step = act_next->step;
  g.nq.r = nullptr;
  g.nq.scale = scale_next;
  g.nq.kc = f8 ? kc_next : nullptr;
  return hip_status(launch_gemm_gelu_quant4(g, stream, f.partial, f.partial_bytes));
}

sq_status sq_gemm_w4a4_fp8(const uint8_t* qx, const float* group_scale, const float* kc, int32_t M,
                           const sq_act_params* act, const sq_weight* w, void* y, int32_t out_dtype, void* workspace,
                           size_t ws_bytes, hipStream_t stream) {
  if (qx == nullptr || group_scale == nullptr || kc == nullptr || y == nullptr) return SQ_ERR_NULL;
  sq_status st = check_weight(w);
  if (st != SQ_OK) return st;
  st = check_act(act, w->K);
  if (st != SQ_OK) return st;
  if (act->act_bits != 4) return SQ_ERR_UNSUPPORTED;
  if (!valid_m(M)) return SQ_ERR_SHAPE;
  if (!a4_fp8_path(M, w->K, w->w_group)) return SQ_ERR_UNSUPPORTED;  // few tokens: packed codes, sq_gemm_w4a4
  if (!valid_out(out_dtype)) return SQ_ERR_UNSUPPORTED;
  if (!aligned(qx, 16) || !aligned(y, 16) || !aligned(group_scale, 4) || !aligned(kc, 4)) return SQ_ERR_ALIGN;
  if (workspace != nullptr && !aligned(workspace, 16)) return SQ_ERR_ALIGN;
  GemmArgs g = gemm_args(qx, group_scale, M, act, w, y, out_dtype);
  g.kc = kc;
  return hip_status(launch_gemm(4, kEpiOut, g, stream, static_cast<float*>(workspace), workspace ? ws_bytes : 0));
}

sq_status sq_gelu_bf16(const uint16_t* x, size_t n, uint16_t* y, hipStream_t stream) {
  if (n > 0 && (x == nullptr || y == nullptr)) return SQ_ERR_NULL;
  if (!aligned(x, 16) || !aligned(y, 16)) return SQ_ERR_ALIGN;
  return hip_status(launch_gelu_bf16(x, n, y, stream));
}

sq_status sq_linear_unfused(const uint16_t* x, int32_t M, const sq_act_params* act, const sq_weight* w,
                            void* y, int32_t out_dtype, void* workspace, size_t ws_bytes,
                            hipStream_t stream) {
  if (x == nullptr || y == nullptr || workspace == nullptr) return SQ_ERR_NULL;
  sq_status st = check_weight(w);
  if (st != SQ_OK) return st;
  st = check_act(act, w->K);
  if (st != SQ_OK) return st;
  if (!valid_m(M)) return SQ_ERR_SHAPE;
  if (!valid_out(out_dtype)) return SQ_ERR_UNSUPPORTED;
  if (!aligned(x, 16) || !aligned(y, 16) || !aligned(workspace, 16)) return SQ_ERR_ALIGN;
  const int32_t K = w->K, N = w->N, bits = act->act_bits;
  if (ws_bytes < unfused_ws_bytes(M, K, N, bits)) return SQ_ERR_WORKSPACE;

  uint8_t* p = static_cast<uint8_t*>(workspace);
  UnfusedArgs u{};
  u.x = x;
  u.tok2stream = act->tok2stream;
  u.gamma = act->gamma;
  u.clip = act->clip;
  u.dinv = act->dinv;
  u.qw = w->qw;
  u.w_scale = w->w_scale;
  u.bias = w->bias;
  u.M = M;
  u.K = K;
  u.N = N;
  u.S = act->num_streams;
  u.step = act->step;
  u.range_mode = act->range_mode;
  u.act_bits = bits;
  u.w_group = w->w_group;
  u.out_dtype = out_dtype;
  const size_t mk4 = round_up(static_cast<size_t>(M) * K * 4);
  const size_t mn4 = round_up(static_cast<size_t>(M) * N * 4);
  const size_t groups = bits == 8 ? 1 : K / kA4Group;
  u.xt = reinterpret_cast<float*>(p);
  p += mk4;
  u.xh = reinterpret_cast<float*>(p);
  p += mk4;
  u.gmax = reinterpret_cast<float*>(p);
  p += round_up(static_cast<size_t>(M) * groups * 4);
  u.qx = p;
  p += round_up(qx_bytes(M, K, bits));
  u.qscale = p;
  p += round_up(act_scale_bytes(M, K, bits));
  u.gemm_out = p;
  p += mn4;
  u.y1 = reinterpret_cast<float*>(p);
  p += mn4;
  u.y2 = reinterpret_cast<float*>(p);
  u.y = y;
  return hip_status(launch_unfused(u, stream));
}

sq_status sq_calib_reference(const uint16_t* x, int32_t M, const float* dinv, const sq_weight* w, double* y_ref,
                             hipStream_t stream) {
  if (x == nullptr || y_ref == nullptr) return SQ_ERR_NULL;
  sq_status st = check_weight(w);
  if (st != SQ_OK) return st;
  if (!valid_m(M)) return SQ_ERR_SHAPE;
  if (!aligned(x, 16) || !aligned(y_ref, 16)) return SQ_ERR_ALIGN;
  if (dinv != nullptr && !aligned(dinv, 16)) return SQ_ERR_ALIGN;
  CalibRefArgs a{x, dinv, w->qw, w->w_scale, nullptr, y_ref, M, w->N, w->K, w->w_group};
  return hip_status(launch_calib_reference(a, stream));
}

sq_status sq_calib_fp_reference(const uint16_t* x, int32_t M, const float* w, int32_t N, int32_t K, double* y_ref,
                                hipStream_t stream) {
  if (x == nullptr || w == nullptr || y_ref == nullptr) return SQ_ERR_NULL;
  if (!valid_m(M) || !valid_k(K) || !valid_n(N)) return SQ_ERR_SHAPE;
  if (!aligned(x, 16) || !aligned(w, 16) || !aligned(y_ref, 16)) return SQ_ERR_ALIGN;
  CalibRefArgs a{x, nullptr, nullptr, nullptr, w, y_ref, M, N, K, 0};
  return hip_status(launch_calib_reference(a, stream));
}

sq_status sq_smooth_scales(const uint16_t* x, int32_t M, const float* w, int32_t N, int32_t K, float alpha, float* d,
                           float* dinv, hipStream_t stream) {
  if (x == nullptr || w == nullptr || d == nullptr || dinv == nullptr) return SQ_ERR_NULL;
  if (!valid_m(M) || !valid_k(K) || N < 1 || N > kMaxN) return SQ_ERR_SHAPE;
  if (!std::isfinite(alpha)) return SQ_ERR_UNSUPPORTED;
  if (!aligned(x, 16) || !aligned(w, 16) || !aligned(d, 4) || !aligned(dinv, 4)) return SQ_ERR_ALIGN;
  if (d == dinv) return SQ_ERR_UNSUPPORTED;
  // the amaxes land in the output buffers, which the last kernel overwrites in place
  sq_status st = hip_status(launch_channel_amax(x, M, w, N, K, reinterpret_cast<uint32_t*>(d),
                                                reinterpret_cast<uint32_t*>(dinv), stream));
  if (st != SQ_OK) return st;
  return hip_status(launch_smooth_scales(reinterpret_cast<const uint32_t*>(d), reinterpret_cast<const uint32_t*>(dinv),
                                         K, alpha, d, dinv, stream));
}

size_t sq_calib_workspace_bytes(int32_t M, int32_t K, int32_t N, int32_t act_bits, int32_t num_streams) {
  if (!valid_m(M) || !valid_k(K) || !valid_n(N) || (act_bits != 8 && act_bits != 4)) return 0;
  if (num_streams < 1 || num_streams > kCalibMaxStreams) return 0;
  return calib_ws_bytes(M, K, N, act_bits, num_streams);
}

sq_status sq_calib_objective(const uint16_t* x, int32_t M, const int32_t* tok2stream, int32_t num_streams,
                             const float* dinv, int32_t act_bits, const sq_weight* w, const double* y_ref,
                             int32_t num_candidates, const float* cand_gamma, const float* cand_clip,
                             const double* omega, double* objective, void* workspace, size_t ws_bytes,
                             hipStream_t stream) {
  if (x == nullptr || tok2stream == nullptr || y_ref == nullptr || cand_gamma == nullptr ||
      cand_clip == nullptr || omega == nullptr || objective == nullptr || workspace == nullptr)
    return SQ_ERR_NULL;
  sq_status st = check_weight(w);
  if (st != SQ_OK) return st;
  if (act_bits != 8 && act_bits != 4) return SQ_ERR_UNSUPPORTED;
  if (!valid_m(M) || num_streams < 1 || num_streams > kCalibMaxStreams || num_candidates < 1 ||
      num_candidates > kCalibMaxCandidates)
    return SQ_ERR_SHAPE;
  if (!aligned(x, 16) || !aligned(y_ref, 16) || !aligned(workspace, 16) || !aligned(tok2stream, 4) ||
      !aligned(cand_gamma, 4) || !aligned(cand_clip, 4) || !aligned(omega, 8) || !aligned(objective, 8))
    return SQ_ERR_ALIGN;
  if (dinv != nullptr && !aligned(dinv, 16)) return SQ_ERR_ALIGN;
  const int32_t K = w->K, N = w->N, S = num_streams;
  if (ws_bytes < calib_ws_bytes(M, K, N, act_bits, S)) return SQ_ERR_WORKSPACE;

  CalibEval e = calib_eval_setup(x, M, tok2stream, S, dinv, act_bits, w, y_ref, omega, workspace);
  st = hip_status(launch_calib_counts(tok2stream, M, S, e.counts, stream));
  if (st != SQ_OK) return st;
  for (int32_t c = 0; c < num_candidates; ++c) {
    st = calib_eval(e, cand_gamma + static_cast<size_t>(c) * S, cand_clip + c, objective + c, stream);
    if (st != SQ_OK) return st;
  }
  return SQ_OK;
}

sq_status sq_calib_search(const uint16_t* x, int32_t M, const int32_t* tok2stream, int32_t num_streams,
                          const float* dinv, int32_t act_bits, const sq_weight* w, const double* y_ref,
                          const double* omega, const sq_calib_search_params* params, float* gamma_out,
                          float* clip_out, double* objective_out, void* workspace, size_t ws_bytes,
                          hipStream_t stream) {
  if (x == nullptr || tok2stream == nullptr || y_ref == nullptr || omega == nullptr || params == nullptr ||
      gamma_out == nullptr || clip_out == nullptr || objective_out == nullptr || workspace == nullptr)
    return SQ_ERR_NULL;
  sq_status st = check_weight(w);
  if (st != SQ_OK) return st;
  if (act_bits != 8 && act_bits != 4) return SQ_ERR_UNSUPPORTED;
  const sq_calib_search_params& p = *params;
  if (!valid_m(M) || num_streams < 1 || num_streams > kCalibSearchMaxStreams || p.rounds < 0 ||
      p.rounds > kCalibSearchMaxRounds)
    return SQ_ERR_SHAPE;
  const bool ok_bounds = std::isfinite(p.gamma_min) && std::isfinite(p.gamma_max) && std::isfinite(p.clip_min) &&
                         std::isfinite(p.clip_max) && std::isfinite(p.clip_init) && std::isfinite(p.log_step) &&
                         p.gamma_min > 0.0f && p.gamma_min <= 1.0f && p.gamma_max >= 1.0f && p.clip_min > 0.0f &&
                         p.clip_min <= p.clip_max && p.log_step > 0.0f && p.log_step <= 64.0f;
  if (!ok_bounds) return SQ_ERR_UNSUPPORTED;
  if (!aligned(x, 16) || !aligned(y_ref, 16) || !aligned(workspace, 16) || !aligned(tok2stream, 4) ||
      !aligned(omega, 8) || !aligned(gamma_out, 4) || !aligned(clip_out, 4) || !aligned(objective_out, 8))
    return SQ_ERR_ALIGN;
  if (dinv != nullptr && !aligned(dinv, 16)) return SQ_ERR_ALIGN;
  const int32_t S = num_streams;
  const size_t base = calib_ws_bytes(M, w->K, w->N, act_bits, S);
  if (ws_bytes < base + search_extra_bytes(S)) return SQ_ERR_WORKSPACE;

  CalibEval e = calib_eval_setup(x, M, tok2stream, S, dinv, act_bits, w, y_ref, omega, workspace);
  SearchWs sw;
  search_extra_bytes(S, &sw, static_cast<uint8_t*>(workspace) + base);
  const SearchBounds b{p.gamma_min, p.gamma_max, p.clip_min, p.clip_max, p.clip_init, p.log_step};
  const int32_t C = 2 * (S + 1);
  st = hip_status(launch_calib_counts(tok2stream, M, S, e.counts, stream));
  if (st != SQ_OK) return st;
  st = hip_status(launch_calib_search_init(b, S, sw.st, sw.u, gamma_out, clip_out, stream));
  if (st != SQ_OK) return st;
  st = calib_eval(e, gamma_out, clip_out, objective_out, stream);
  if (st != SQ_OK) return st;
  for (int32_t r = 0; r < p.rounds; ++r) {
    st = hip_status(launch_calib_propose(b, S, e.counts, sw.st, sw.u, sw.cand_u, sw.cand_v, sw.cand_gamma,
                                         sw.cand_clip, stream));
    if (st != SQ_OK) return st;
    for (int32_t c = 0; c < C; ++c) {
      st = calib_eval(e, sw.cand_gamma + static_cast<size_t>(c) * S, sw.cand_clip + c, sw.cand_obj + c, stream);
      if (st != SQ_OK) return st;
    }
    st = hip_status(launch_calib_select(S, sw.cand_obj, sw.cand_u, sw.cand_v, sw.cand_gamma, sw.cand_clip, sw.st,
                                        sw.u, gamma_out, clip_out, objective_out, stream));
    if (st != SQ_OK) return st;
  }
  return SQ_OK;
}

size_t sq_calib_scaling_workspace_bytes(int32_t M, int32_t K, int32_t N, int32_t w_group, int32_t act_bits,
                                        int32_t num_regions) {
  if (w_group < kKTile || w_group % kKTile != 0 || !valid_k(K) || K % w_group != 0) return 0;
  const size_t base = sq_calib_workspace_bytes(M, K, N, act_bits, num_regions);
  return base == 0 ? 0 : base + scaling_extra_bytes(K, N, w_group, num_regions);
}

sq_status sq_calib_scaling_objective(const uint16_t* x, int32_t M, const int32_t* region, int32_t num_regions,
                                     const double* region_weight, const float* w, int32_t N, int32_t K,
                                     int32_t w_group, int32_t act_bits, const double* y_ref, int32_t num_alphas,
                                     const float* alphas, double* objective, void* workspace, size_t ws_bytes,
                                     hipStream_t stream) {
  if (x == nullptr || region == nullptr || region_weight == nullptr || w == nullptr || y_ref == nullptr ||
      alphas == nullptr || objective == nullptr || workspace == nullptr)
    return SQ_ERR_NULL;
  if (act_bits != 8 && act_bits != 4) return SQ_ERR_UNSUPPORTED;
  if (!valid_m(M) || !valid_k(K) || !valid_n(N) || num_regions < 1 || num_regions > kCalibMaxStreams ||
      num_alphas < 1 || num_alphas > kCalibMaxCandidates)
    return SQ_ERR_SHAPE;
  if (w_group < kKTile || w_group % kKTile != 0 || K % w_group != 0) return SQ_ERR_UNSUPPORTED;
  for (int32_t i = 0; i < num_alphas; ++i)
    if (!std::isfinite(alphas[i])) return SQ_ERR_UNSUPPORTED;
  if (!aligned(x, 16) || !aligned(w, 16) || !aligned(y_ref, 16) || !aligned(workspace, 16) || !aligned(region, 4) ||
      !aligned(region_weight, 8) || !aligned(objective, 8))
    return SQ_ERR_ALIGN;
  const int32_t R = num_regions;
  const size_t base = calib_ws_bytes(M, K, N, act_bits, R);
  if (ws_bytes < base + scaling_extra_bytes(K, N, w_group, R)) return SQ_ERR_WORKSPACE;
  ScalingWs sw;
  scaling_extra_bytes(K, N, w_group, R, &sw, static_cast<uint8_t*>(workspace) + base);
  // Q(D W) lands in the workspace; Eq. 7 has no gain: a one-step table of ones
  sq_weight wt{sw.qw, sw.w_scale, nullptr, N, K, w_group};
  CalibEval e = calib_eval_setup(x, M, region, R, sw.dinv, act_bits, &wt, y_ref, region_weight, workspace);
  sq_status st = hip_status(launch_calib_counts(region, M, R, e.counts, stream));
  if (st != SQ_OK) return st;
  st = hip_status(launch_fill_f32(sw.ones, R, 1.0f, stream));
  if (st != SQ_OK) return st;
  st = hip_status(launch_channel_amax(x, M, w, N, K, sw.ax, sw.aw, stream));
  if (st != SQ_OK) return st;
  for (int32_t i = 0; i < num_alphas; ++i) {
    st = hip_status(launch_smooth_scales(sw.ax, sw.aw, K, alphas[i], sw.d, sw.dinv, stream));
    if (st != SQ_OK) return st;
    PackArgs pk{w, sw.d, sw.qw, sw.w_scale, N, K, w_group};
    st = hip_status(launch_pack_weights(pk, stream));
    if (st != SQ_OK) return st;
    st = calib_eval_range(e, sw.ones, nullptr, SQ_RANGE_DYNAMIC, objective + i, stream);
    if (st != SQ_OK) return st;
  }
  return SQ_OK;
}

size_t sq_calib_search_workspace_bytes(int32_t M, int32_t K, int32_t N, int32_t act_bits, int32_t num_streams) {
  if (num_streams > kCalibSearchMaxStreams) return 0;
  const size_t base = sq_calib_workspace_bytes(M, K, N, act_bits, num_streams);
  return base == 0 ? 0 : base + search_extra_bytes(num_streams);
}

size_t sq_probe_mfma_i8_sink_bytes(void) { return static_cast<size_t>(mfma_probe_workgroups()) * 256 * 4; }

sq_status sq_probe_mfma_i8(int32_t shape, int32_t iters, int32_t random_operands, int32_t fold, int32_t* sink,
                           size_t sink_bytes, hipStream_t stream) {
  if (sink == nullptr) return SQ_ERR_NULL;
  if (shape != 32 && shape != 16) return SQ_ERR_UNSUPPORTED;
  if (iters < 1 || iters > (1 << 24)) return SQ_ERR_SHAPE;
  if (sink_bytes < sq_probe_mfma_i8_sink_bytes()) return SQ_ERR_WORKSPACE;
  if (!aligned(sink, 4)) return SQ_ERR_ALIGN;
  return hip_status(launch_mfma_probe(sink, shape, iters, random_operands != 0, fold != 0, stream));
}

sq_status sq_probe_mfma_f8f6(int32_t format, int32_t iters, int32_t random_operands, int32_t fold, int32_t* sink,
                             size_t sink_bytes, hipStream_t stream) {
  if (sink == nullptr) return SQ_ERR_NULL;
  if (format != 8 && format != 6) return SQ_ERR_UNSUPPORTED;
  if (iters < 1 || iters > (1 << 24)) return SQ_ERR_SHAPE;
  if (sink_bytes < sq_probe_mfma_i8_sink_bytes()) return SQ_ERR_WORKSPACE;
  if (!aligned(sink, 4)) return SQ_ERR_ALIGN;
  return hip_status(launch_mfma_probe_f8f6(sink, format, iters, random_operands != 0, fold != 0, stream));
}

sq_status sq_debug_block_acc_i32(const void* qx, int32_t M, int32_t act_bits, const sq_weight* w,
                                 int32_t* acc_out, hipStream_t stream) {
  if (qx == nullptr || acc_out == nullptr) return SQ_ERR_NULL;
  sq_status st = check_weight(w);
  if (st != SQ_OK) return st;
  if (act_bits != 8 && act_bits != 4) return SQ_ERR_UNSUPPORTED;
  if (!valid_m(M)) return SQ_ERR_SHAPE;
  if (!aligned(qx, 16) || !aligned(acc_out, 4)) return SQ_ERR_ALIGN;
  GemmArgs g = gemm_args(qx, nullptr, M, nullptr, w, acc_out, SQ_OUT_F32);
  return hip_status(launch_gemm(act_bits, kEpiDump, g, stream));
}

}  // extern "C"
