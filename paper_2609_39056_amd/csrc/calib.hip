// Calibration.  Activation calibration (Sec. 4.3, Eq. 9): the reconstruction
// error of one linear under a candidate (gain per stream, shared threshold),
// weighted per stream by omega_s / n_s, and a constrained search over
// candidates.  Shared scaling (Sec. 4.2, Eq. 7): the same error against the
// full-precision product for a family of channel scalings D.
//
//   - calib_reference_kernel<false>: the target X~ W^ in fp64, X~ = fp32(x) *
//     dinv (the quantizer's first step) and W^ = code * Delta_W.  Every
//     product is exact in fp64 (24 x 15 significant bits), so the kernel
//     differs from any other fp64 evaluation only in the order of its K sums.
//     128 x 128 output tiles, each thread 8 x 8 of them, K staged 16 at a time
//     through LDS already widened to fp64.  Computed once per linear.
//     calib_reference_kernel<true>: the same with fp32 W (the target X W of
//     Eq. 7; products of 8 x 24 significant bits, exact).
//   - channel_amax_kernel, smooth_scale_kernel: the per-channel maxima of |X|
//     and |W| and the family d = amax|X|^alpha / amax|W|^(1 - alpha) of Eq. 7.
//   - calib_count_kernel: n_s, the tokens of every stream (LDS histogram per
//     workgroup, one global add per non-empty bin).
//   - calib_row_error_kernel: e_i = omega_s(i) / n_s(i) * sum_j (y_ij - ref_ij)^2
//     for the candidate's fp32 output y, one wave per row, fixed order.
//   - calib_sum_kernel: L = sum_i e_i in one workgroup, fixed order.
// The candidate's output itself comes from the fused linear (no bias; STATIC
// with the candidate's one-step table for Eq. 9, DYNAMIC with unit gains for
// Eq. 7), so the objective measures the arithmetic that runs.
#include "sq_internal.h"

namespace sq {
namespace {

constexpr int kRefTile = 128;  // output rows and columns per workgroup
constexpr int kRefKc = 16;     // K per LDS stage

// FPW: the weight operand is fp32 W [N][K] itself (the full-precision target
// of Eq. 7, no D^-1); otherwise packed codes times their fp16 steps.
template <bool FPW>
__global__ __launch_bounds__(256) void calib_reference_kernel(const uint16_t* __restrict__ x,
                                                              const float* __restrict__ dinv,
                                                              const uint8_t* __restrict__ qw,
                                                              const uint16_t* __restrict__ w_scale,
                                                              const float* __restrict__ wf,
                                                              double* __restrict__ y, int32_t M, int32_t N,
                                                              int32_t K, int32_t w_group, int32_t tiles_n,
                                                              size_t n_tiles) {
  const size_t wg = flat_wg();
  if (wg >= n_tiles) return;
  const int64_t m0 = static_cast<int64_t>(wg / tiles_n) * kRefTile;
  const int32_t n0 = static_cast<int32_t>(wg % tiles_n) * kRefTile;
  __shared__ double xs[kRefKc][kRefTile];
  __shared__ double ws[kRefKc][kRefTile];

  const int t = threadIdx.x;
  const int tx = t & 15, ty = t >> 4;
  // staging: thread t fills row / column t/2 of the tile, channels 8*(t%2) .. +7 of the stage
  const int sr = t >> 1, sh = t & 1;
  const int64_t xm = m0 + sr;
  const bool xin = xm < M;
  const int32_t wn = n0 + sr;
  const bool win = wn < N;
  const uint16_t* xrow = x + (xin ? xm : 0) * static_cast<int64_t>(K);
  const uint8_t* wrow = FPW ? nullptr : qw + static_cast<size_t>(win ? wn : 0) * (K / 2);
  const float* wfrow = FPW ? wf + static_cast<size_t>(win ? wn : 0) * K : nullptr;

  double acc[8][8];
#pragma unroll
  for (int r = 0; r < 8; ++r)
#pragma unroll
    for (int c = 0; c < 8; ++c) acc[r][c] = 0.0;

  for (int32_t k0 = 0; k0 < K; k0 += kRefKc) {
    const int32_t kb = k0 + sh * 8;
    uint4 xv = make_uint4(0u, 0u, 0u, 0u);
    if (xin) xv = *reinterpret_cast<const uint4*>(xrow + kb);
    float d[8];
    if (dinv != nullptr) {
      const float4 d0 = *reinterpret_cast<const float4*>(dinv + kb);
      const float4 d1 = *reinterpret_cast<const float4*>(dinv + kb + 4);
      d[0] = d0.x; d[1] = d0.y; d[2] = d0.z; d[3] = d0.w;
      d[4] = d1.x; d[5] = d1.y; d[6] = d1.z; d[7] = d1.w;
    }
    const uint32_t xw[4] = {xv.x, xv.y, xv.z, xv.w};
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const float xf = bf16_to_f32((xw[j >> 1] >> (16 * (j & 1))) & 0xFFFFu);
      xs[sh * 8 + j][sr] = static_cast<double>(dinv != nullptr ? xf * d[j] : xf);
    }
    if constexpr (FPW) {
      float4 w0 = make_float4(0.f, 0.f, 0.f, 0.f), w1 = w0;
      if (win) {
        w0 = *reinterpret_cast<const float4*>(wfrow + kb);
        w1 = *reinterpret_cast<const float4*>(wfrow + kb + 4);
      }
      const float wv[8] = {w0.x, w0.y, w0.z, w0.w, w1.x, w1.y, w1.z, w1.w};
#pragma unroll
      for (int j = 0; j < 8; ++j) ws[sh * 8 + j][sr] = static_cast<double>(wv[j]);
    } else {
      // 8 codes kb .. kb+7 sit in one dword: byte b holds code kb+b (low
      // nibble) and code kb+b+4 (high nibble)
      uint32_t p = 0u;
      double step = 0.0;
      if (win) {
        p = *reinterpret_cast<const uint32_t*>(wrow + kb / 2);
        step = static_cast<double>(f16_to_f32(w_scale[static_cast<size_t>(kb / w_group) * N + wn]));
      }
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        const int lo = static_cast<int32_t>(p << (28 - 8 * b)) >> 28;
        const int hi = static_cast<int32_t>(p << (24 - 8 * b)) >> 28;
        ws[sh * 8 + b][sr] = static_cast<double>(lo) * step;
        ws[sh * 8 + b + 4][sr] = static_cast<double>(hi) * step;
      }
    }
    __syncthreads();
#pragma unroll 4
    for (int kk = 0; kk < kRefKc; ++kk) {
      double a[8], bv[8];
#pragma unroll
      for (int r = 0; r < 8; ++r) a[r] = xs[kk][ty + 16 * r];
#pragma unroll
      for (int c = 0; c < 8; ++c) bv[c] = ws[kk][tx + 16 * c];
#pragma unroll
      for (int r = 0; r < 8; ++r)
#pragma unroll
        for (int c = 0; c < 8; ++c) acc[r][c] = fma(a[r], bv[c], acc[r][c]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int r = 0; r < 8; ++r) {
    const int64_t m = m0 + ty + 16 * r;
    if (m >= M) continue;
#pragma unroll
    for (int c = 0; c < 8; ++c) {
      const int32_t n = n0 + tx + 16 * c;
      if (n < N) y[m * N + n] = acc[r][c];
    }
  }
}

__global__ __launch_bounds__(256) void calib_zero_kernel(int32_t* __restrict__ counts, int32_t S) {
  for (int32_t s = blockIdx.x * 256 + threadIdx.x; s < S; s += gridDim.x * 256) counts[s] = 0;
}

__global__ __launch_bounds__(256) void calib_count_kernel(const int32_t* __restrict__ tok2stream, int32_t M,
                                                          int32_t S, int32_t* __restrict__ counts) {
  __shared__ int32_t bins[kCalibMaxStreams];
  for (int32_t s = threadIdx.x; s < S; s += 256) bins[s] = 0;
  __syncthreads();
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x; i < M;
       i += static_cast<int64_t>(gridDim.x) * 256) {
    const int32_t s = tok2stream[i];
    if (static_cast<uint32_t>(s) < static_cast<uint32_t>(S)) atomicAdd(&bins[s], 1);
  }
  __syncthreads();
  for (int32_t s = threadIdx.x; s < S; s += 256)
    if (bins[s] != 0) atomicAdd(&counts[s], bins[s]);
}

__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// One wave per row; four rows per workgroup.
__global__ __launch_bounds__(256) void calib_row_error_kernel(const float* __restrict__ yq,
                                                              const double* __restrict__ ref,
                                                              const int32_t* __restrict__ tok2stream,
                                                              const int32_t* __restrict__ counts,
                                                              const double* __restrict__ omega, int32_t M,
                                                              int32_t N, int32_t S, double* __restrict__ err) {
  const int64_t i = static_cast<int64_t>(flat_wg()) * 4 + (threadIdx.x >> 6);
  if (i >= M) return;
  const int lane = threadIdx.x & 63;
  const float4* yr = reinterpret_cast<const float4*>(yq + i * N);
  const double2* rr = reinterpret_cast<const double2*>(ref + i * N);
  double acc = 0.0;
#pragma unroll 4
  for (int32_t j = lane; j < N / 4; j += 64) {
    const float4 a = yr[j];
    const double2 b0 = rr[2 * j], b1 = rr[2 * j + 1];
    const double e0 = static_cast<double>(a.x) - b0.x, e1 = static_cast<double>(a.y) - b0.y;
    const double e2 = static_cast<double>(a.z) - b1.x, e3 = static_cast<double>(a.w) - b1.y;
    acc = fma(e0, e0, acc);
    acc = fma(e1, e1, acc);
    acc = fma(e2, e2, acc);
    acc = fma(e3, e3, acc);
  }
  acc = wave_sum(acc);
  if (lane == 0) {
    const int32_t s = tok2stream[i];
    double w = 0.0;
    if (static_cast<uint32_t>(s) < static_cast<uint32_t>(S)) w = omega[s] / static_cast<double>(counts[s]);
    err[i] = w * acc;
  }
}

__global__ __launch_bounds__(256) void calib_sum_kernel(const double* __restrict__ err, int32_t M,
                                                        double* __restrict__ out) {
  __shared__ double part[4];
  double acc = 0.0;
  for (int64_t i = threadIdx.x; i < M; i += 256) acc += err[i];
  acc = wave_sum(acc);
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0) *out = (part[0] + part[1]) + (part[2] + part[3]);
}

// ---------------------------------------------------------------- shared channel scaling (Eq. 7)
// Per-channel absolute maxima by atomic max on the bits of |v| (non-negative
// floats order like their bit patterns; the result does not depend on the
// order), then d_k = amax|X_k|^alpha / amax|W_k|^(1 - alpha) in fp64, clamped
// to [2^-6, 2^6], and dinv = 1 / d in fp32.
__global__ __launch_bounds__(256) void calib_fill_kernel(float* __restrict__ p, int32_t n, float v) {
  for (int32_t i = blockIdx.x * 256 + threadIdx.x; i < n; i += gridDim.x * 256) p[i] = v;
}

__global__ __launch_bounds__(256) void calib_zero_u32_kernel(uint32_t* __restrict__ p, int32_t n) {
  for (int32_t i = blockIdx.x * 256 + threadIdx.x; i < n; i += gridDim.x * 256) p[i] = 0u;
}

// A workgroup covers 32 x CH channels (CH = 8 bf16 or 4 fp32: one 16-byte
// load per row) and a range of rows (grid.y); its eight row lanes take every
// eighth row, meet in LDS, and one atomic max per channel leaves the
// workgroup.
constexpr int kAmaxLanes = 32;
template <bool BF16>
__global__ __launch_bounds__(256) void channel_amax_kernel(const void* __restrict__ src, int64_t rows, int32_t K,
                                                           int64_t rows_per_block, uint32_t* __restrict__ amax) {
  constexpr int CH = BF16 ? 8 : 4;
  constexpr int WCH = kAmaxLanes * CH;  // channels per workgroup
  __shared__ uint32_t red[8][WCH];
  const int cl = threadIdx.x % kAmaxLanes, rl = threadIdx.x / kAmaxLanes;
  const int32_t k0 = blockIdx.x * WCH + cl * CH;
  const int64_t r0 = static_cast<int64_t>(blockIdx.y) * rows_per_block;
  const int64_t r1 = min(rows, r0 + rows_per_block);
  const size_t row_bytes = static_cast<size_t>(K) * (BF16 ? 2 : 4);
  uint32_t m[CH];
#pragma unroll
  for (int c = 0; c < CH; ++c) m[c] = 0u;
  if (k0 < K) {
    const uint8_t* base = static_cast<const uint8_t*>(src) + static_cast<size_t>(k0) * (BF16 ? 2 : 4);
#pragma unroll 4
    for (int64_t r = r0 + rl; r < r1; r += 8) {
      const uint4 v = *reinterpret_cast<const uint4*>(base + static_cast<size_t>(r) * row_bytes);
      const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int c = 0; c < CH; ++c) {
        const uint32_t b = BF16 ? ((w[c >> 1] >> (16 * (c & 1))) & 0x7FFFu) << 16 : w[c] & 0x7FFFFFFFu;
        m[c] = max(m[c], b);
      }
    }
  }
#pragma unroll
  for (int c = 0; c < CH; ++c) red[rl][cl * CH + c] = m[c];
  __syncthreads();
  if (threadIdx.x < WCH) {
    uint32_t v = red[0][threadIdx.x];
#pragma unroll
    for (int i = 1; i < 8; ++i) v = max(v, red[i][threadIdx.x]);
    const int32_t k = blockIdx.x * WCH + threadIdx.x;
    if (k < K && v != 0u) atomicMax(&amax[k], v);
  }
}

__global__ __launch_bounds__(256) void smooth_scale_kernel(const uint32_t* __restrict__ ax_bits,
                                                           const uint32_t* __restrict__ aw_bits, int32_t K,
                                                           float alpha, float* __restrict__ d,
                                                           float* __restrict__ dinv) {
  const int32_t k = blockIdx.x * 256 + threadIdx.x;
  if (k >= K) return;
  const double ax = static_cast<double>(__uint_as_float(ax_bits[k]));
  const double aw = static_cast<double>(__uint_as_float(aw_bits[k]));
  const double a = static_cast<double>(alpha);
  double v = 1.0;
  if (ax > 0.0 && aw > 0.0) v = pow(ax, a) / pow(aw, 1.0 - a);
  const float dk = static_cast<float>(fmin(fmax(v, 0.015625), 64.0));
  d[k] = dk;
  dinv[k] = 1.0f / dk;
}

// ---------------------------------------------------------------- constrained search
// Compass search over (log gamma_1 .. log gamma_S, log c).  State in device
// memory: st = {unused, h, log c}, u = the incumbent's log gains, and the
// caller's gamma / clip / objective outputs hold the incumbent's evaluated
// values.  Candidate j of a round moves coordinate j/2 (the gains, then the
// threshold) by +h (j even) or -h (j odd).

__device__ __forceinline__ double clampd(double v, double lo, double hi) { return fmin(fmax(v, lo), hi); }
__device__ __forceinline__ float clampf_(float v, float lo, float hi) { return fminf(fmaxf(v, lo), hi); }

__global__ __launch_bounds__(64) void calib_search_init_kernel(SearchBounds b, int32_t S, double* st, double* u,
                                                               float* gamma, float* clip) {
  for (int32_t s = threadIdx.x; s < S; s += 64) {
    u[s] = 0.0;
    gamma[s] = 1.0f;
  }
  if (threadIdx.x == 0) {
    const float c = clampf_(b.clip_init, b.clip_min, b.clip_max);
    clip[0] = c;
    st[0] = 0.0;
    st[1] = static_cast<double>(b.log_step);
    st[2] = log(static_cast<double>(c));
  }
}

// One thread per candidate (C = 2 (S + 1) <= 256).  A gain step is projected
// onto lo <= u_s <= hi, sum_s n_s u_s = 0 (nearest point in the token-
// weighted norm: u_s = clamp(w_s - lam) for streams with tokens, lam by 64
// bisection halvings in fp64); a threshold step is clamped to the log bounds.
__global__ __launch_bounds__(256) void calib_propose_kernel(SearchBounds b, int32_t S, const int32_t* counts,
                                                            const double* st, const double* u, double* cand_u,
                                                            double* cand_v, float* cand_gamma, float* cand_clip) {
  const int32_t C = 2 * (S + 1);
  const int32_t j = threadIdx.x;
  if (j >= C) return;
  const int32_t d = j >> 1;
  const double step = (j & 1) ? -st[1] : st[1];
  const double lo = log(static_cast<double>(b.gamma_min)), hi = log(static_cast<double>(b.gamma_max));
  double* uj = cand_u + static_cast<size_t>(j) * S;
  double vc = st[2];
  if (d < S) {
    bool any = false;
    double wmin = 0.0, wmax = 0.0;
    for (int32_t s = 0; s < S; ++s) {
      const double w = u[s] + (s == d ? step : 0.0);
      if (counts[s] > 0) {
        wmin = any ? fmin(wmin, w) : w;
        wmax = any ? fmax(wmax, w) : w;
        any = true;
      }
    }
    double lam = 0.0;
    if (any) {
      double a = wmin - hi, c = wmax - lo;
      for (int it = 0; it < 64; ++it) {
        const double mid = 0.5 * (a + c);
        double f = 0.0;
        for (int32_t s = 0; s < S; ++s) {
          if (counts[s] <= 0) continue;
          const double w = u[s] + (s == d ? step : 0.0);
          f += static_cast<double>(counts[s]) * clampd(w - mid, lo, hi);
        }
        if (f > 0.0)
          a = mid;
        else
          c = mid;
      }
      lam = 0.5 * (a + c);
    }
    for (int32_t s = 0; s < S; ++s) {
      const double w = u[s] + (s == d ? step : 0.0);
      uj[s] = counts[s] > 0 ? clampd(w - lam, lo, hi) : clampd(w, lo, hi);
    }
  } else {
    for (int32_t s = 0; s < S; ++s) uj[s] = u[s];
    vc = clampd(vc + step, log(static_cast<double>(b.clip_min)), log(static_cast<double>(b.clip_max)));
  }
  for (int32_t s = 0; s < S; ++s)
    cand_gamma[static_cast<size_t>(j) * S + s] =
        clampf_(static_cast<float>(exp(uj[s])), b.gamma_min, b.gamma_max);
  cand_v[j] = vc;
  cand_clip[j] = clampf_(static_cast<float>(exp(vc)), b.clip_min, b.clip_max);
}

// The first candidate with the smallest objective replaces the incumbent if
// strictly better; otherwise the step halves.
__global__ __launch_bounds__(64) void calib_select_kernel(int32_t S, const double* cand_obj, const double* cand_u,
                                                          const double* cand_v, const float* cand_gamma,
                                                          const float* cand_clip, double* st, double* u,
                                                          float* gamma, float* clip, double* objective) {
  const int32_t C = 2 * (S + 1);
  int32_t best = 0;
  for (int32_t j = 1; j < C; ++j)
    if (cand_obj[j] < cand_obj[best]) best = j;
  const bool better = cand_obj[best] < objective[0];
  __syncthreads();  // every thread has read objective[0] before it changes
  if (better) {
    for (int32_t s = threadIdx.x; s < S; s += 64) {
      u[s] = cand_u[static_cast<size_t>(best) * S + s];
      gamma[s] = cand_gamma[static_cast<size_t>(best) * S + s];
    }
    if (threadIdx.x == 0) {
      st[2] = cand_v[best];
      clip[0] = cand_clip[best];
      objective[0] = cand_obj[best];
    }
  } else if (threadIdx.x == 0) {
    st[1] = 0.5 * st[1];
  }
}

}  // namespace

hipError_t launch_calib_search_init(const SearchBounds& b, int32_t S, double* st, double* u, float* gamma,
                                    float* clip, hipStream_t s) {
  hipLaunchKernelGGL(calib_search_init_kernel, dim3(1), dim3(64), 0, s, b, S, st, u, gamma, clip);
  return hipGetLastError();
}

hipError_t launch_calib_propose(const SearchBounds& b, int32_t S, const int32_t* counts, const double* st,
                                const double* u, double* cand_u, double* cand_v, float* cand_gamma,
                                float* cand_clip, hipStream_t s) {
  hipLaunchKernelGGL(calib_propose_kernel, dim3(1), dim3(256), 0, s, b, S, counts, st, u, cand_u, cand_v,
                     cand_gamma, cand_clip);
  return hipGetLastError();
}

hipError_t launch_calib_select(int32_t S, const double* cand_obj, const double* cand_u, const double* cand_v,
                               const float* cand_gamma, const float* cand_clip, double* st, double* u,
                               float* gamma, float* clip, double* objective, hipStream_t s) {
  hipLaunchKernelGGL(calib_select_kernel, dim3(1), dim3(64), 0, s, S, cand_obj, cand_u, cand_v, cand_gamma,
                     cand_clip, st, u, gamma, clip, objective);
  return hipGetLastError();
}

hipError_t launch_calib_reference(const CalibRefArgs& a, hipStream_t s) {
  const int32_t tiles_n = (a.N + kRefTile - 1) / kRefTile;
  const size_t n_tiles = static_cast<size_t>((a.M + kRefTile - 1) / kRefTile) * tiles_n;
  if (a.wf != nullptr)
    hipLaunchKernelGGL(calib_reference_kernel<true>, wg_grid(n_tiles), dim3(256), 0, s, a.x, nullptr, nullptr,
                       nullptr, a.wf, a.y, a.M, a.N, a.K, 0, tiles_n, n_tiles);
  else
    hipLaunchKernelGGL(calib_reference_kernel<false>, wg_grid(n_tiles), dim3(256), 0, s, a.x, a.dinv, a.qw,
                       a.w_scale, nullptr, a.y, a.M, a.N, a.K, a.w_group, tiles_n, n_tiles);
  return hipGetLastError();
}

namespace {
void launch_amax(bool bf16, const void* src, int64_t rows, int32_t K, uint32_t* amax, hipStream_t s) {
  const int64_t rpb = 256;  // rows per workgroup: one atomic per channel per 256 rows
  const int64_t yb = (rows + rpb - 1) / rpb;
  const int64_t ybc = yb < 65535 ? yb : 65535;
  const int64_t per = (rows + ybc - 1) / ybc;
  const int wch = kAmaxLanes * (bf16 ? 8 : 4);
  const dim3 grid((K + wch - 1) / wch, static_cast<unsigned>(ybc));
  if (bf16)
    hipLaunchKernelGGL(channel_amax_kernel<true>, grid, dim3(256), 0, s, src, rows, K, per, amax);
  else
    hipLaunchKernelGGL(channel_amax_kernel<false>, grid, dim3(256), 0, s, src, rows, K, per, amax);
}
}  // namespace

hipError_t launch_channel_amax(const uint16_t* x, int32_t M, const float* w, int32_t N, int32_t K,
                               uint32_t* ax_bits, uint32_t* aw_bits, hipStream_t s) {
  hipLaunchKernelGGL(calib_zero_u32_kernel, dim3((K + 255) / 256), dim3(256), 0, s, ax_bits, K);
  hipLaunchKernelGGL(calib_zero_u32_kernel, dim3((K + 255) / 256), dim3(256), 0, s, aw_bits, K);
  launch_amax(true, x, M, K, ax_bits, s);
  launch_amax(false, w, N, K, aw_bits, s);
  return hipGetLastError();
}

hipError_t launch_smooth_scales(const uint32_t* ax_bits, const uint32_t* aw_bits, int32_t K, float alpha, float* d,
                                float* dinv, hipStream_t s) {
  hipLaunchKernelGGL(smooth_scale_kernel, dim3((K + 255) / 256), dim3(256), 0, s, ax_bits, aw_bits, K, alpha, d,
                     dinv);
  return hipGetLastError();
}

hipError_t launch_fill_f32(float* p, int32_t n, float v, hipStream_t s) {
  hipLaunchKernelGGL(calib_fill_kernel, dim3((n + 255) / 256), dim3(256), 0, s, p, n, v);
  return hipGetLastError();
}

hipError_t launch_calib_counts(const int32_t* tok2stream, int32_t M, int32_t S, int32_t* counts, hipStream_t s) {
  hipLaunchKernelGGL(calib_zero_kernel, dim3((S + 255) / 256), dim3(256), 0, s, counts, S);
  const int64_t want = (static_cast<int64_t>(M) + 4095) / 4096;  // about 16 rows per thread
  const int grid = static_cast<int>(want < 1024 ? want : 1024);
  hipLaunchKernelGGL(calib_count_kernel, dim3(grid), dim3(256), 0, s, tok2stream, M, S, counts);
  return hipGetLastError();
}

hipError_t launch_calib_error(const float* yq, const double* ref, const int32_t* tok2stream,
                              const int32_t* counts, const double* omega, int32_t M, int32_t N, int32_t S,
                              double* err, double* out, hipStream_t s) {
  const size_t wgs = (static_cast<size_t>(M) + 3) / 4;
  hipLaunchKernelGGL(calib_row_error_kernel, wg_grid(wgs), dim3(256), 0, s, yq, ref, tok2stream, counts, omega,
                     M, N, S, err);
  hipLaunchKernelGGL(calib_sum_kernel, dim3(1), dim3(256), 0, s, err, M, out);
  return hipGetLastError();
}

}  // namespace sq
