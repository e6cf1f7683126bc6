// Stage 2: Wavelet Temporal Allocator (Sec. 3.2.2 gate and frame filter,
// Eq. (9)-(11)) and the integer frame budgets (Eq. (16) under Eq. (5)).
//
// The whole stage is a few fp64 operations per frame, so it runs as ONE
// workgroup with every array in LDS: one wave when T <= 64 (no cross-wave
// synchronisation at all), 256 threads up to T = 256, 1024 beyond.  Steps:
//   gamma  = min-max(delta) over all T frames (0 if all equal);
//   M      = {0} U {t >= 1 : delta_t >= tau}, compacted in temporal order;
//   WTA    = J levels of orthonormal Haar analysis of r over M (odd lengths
//            repeat the last sample), detail level j multiplied by gamma
//            pair-averaged j times, then synthesis back to length |M|;
//   budget = capped largest remainder on w = max(r~, 0): quotas
//            R * w_m / sum(w); frames reaching H*W are fixed there and the
//            rest re-apportioned; leftover tokens go to the largest
//            fractional parts (ties: smaller frame index); uniform weights if
//            every w is 0; every frame full when B >= |M| * H * W.
#include "wz_internal.h"

namespace wz {
namespace {

constexpr int kTMax = kMaxFrames;
constexpr int kMaxLevels = 16;

enum : unsigned char { kIdle = 0, kActive = 1, kFull = 2 };

struct Shared {
  double a[2][kTMax];              // approximation (ping-pong), then r~ in a[0]
  double g[2][kTMax];              // gate pooled alongside (ping-pong); g[0] reused for weights
  double det[kTMax + kMaxLevels];  // gated detail coefficients of every level
  int idx[kTMax];                  // frame index of each retained position
  int n[kTMax];                    // budget of each retained position
  int fb[kTMax];                   // budget of each frame
  unsigned char state[kTMax];
  double dred[16];
  int ired[16];
  int lens[kMaxLevels];
  int doffs[kMaxLevels];
};

template <int NT>
__device__ double bsum(double v, Shared& sh) {
  v = wave_sum_f64(v);
  if (NT == kWave) return v;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) sh.dred[wave] = v;
  __syncthreads();
  double s = 0.0;
#pragma unroll
  for (int i = 0; i < NT / kWave; ++i) s += sh.dred[i];
  return s;
}

template <int NT>
__device__ double bminmax(double v, bool want_max, Shared& sh) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) {
    const double o = __shfl_xor(v, m, kWave);
    v = want_max ? fmax(v, o) : fmin(v, o);
  }
  if (NT == kWave) return v;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) sh.dred[wave] = v;
  __syncthreads();
  double r = sh.dred[0];
#pragma unroll
  for (int i = 1; i < NT / kWave; ++i) r = want_max ? fmax(r, sh.dred[i]) : fmin(r, sh.dred[i]);
  return r;
}

template <int NT>
__device__ int bsum_int(int v, Shared& sh) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, kWave);
  if (NT == kWave) return v;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) sh.ired[wave] = v;
  __syncthreads();
  int s = 0;
#pragma unroll
  for (int i = 0; i < NT / kWave; ++i) s += sh.ired[i];
  return s;
}

// Exclusive prefix sum over the block in thread order; `total` gets the sum.
template <int NT>
__device__ int bscan_excl(int v, int& total, Shared& sh) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int inc = v;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const int o = __shfl_up(inc, d, kWave);
    if (lane >= d) inc += o;
  }
  if (NT == kWave) {
    total = __shfl(inc, 63, kWave);
    return inc - v;
  }
  __syncthreads();
  if (lane == 63) sh.ired[wave] = inc;
  __syncthreads();
  int before = 0;
  total = 0;
#pragma unroll
  for (int i = 0; i < NT / kWave; ++i) {
    if (i < wave) before += sh.ired[i];
    total += sh.ired[i];
  }
  return before + inc - v;
}

// NT threads handle up to TV frames; thread tid owns frames tid*kPer .. tid*kPer+kPer-1.
template <int NT, int TV>
__global__ __launch_bounds__(NT) void k_temporal_budget(const float* __restrict__ rel,
                                                        const float* __restrict__ delta, int T, int N,
                                                        long long B, int levels, float tau,
                                                        int32_t* __restrict__ budget,
                                                        int32_t* __restrict__ offset,
                                                        float* __restrict__ rel_rect) {
  constexpr int kPer = (TV + NT - 1) / NT;  // frames per thread (contiguous run)
  static_assert(kPer <= 32 && TV <= kTMax, "frame mask holds 32 frames per thread");
  __shared__ Shared sh;
  const int tid = threadIdx.x;
  const double inv_sqrt2 = 0.70710678118654752440;

  // ---- gamma = min-max(delta); retained set M (thread tid owns frames tid*kPer ..) ----
  double dv[kPer], lo = INFINITY, hi = -INFINITY;
#pragma unroll
  for (int k = 0; k < kPer; ++k) {
    const int t = tid * kPer + k;
    dv[k] = t < T ? double(delta[t]) : 0.0;
    if (t < T) { lo = fmin(lo, dv[k]); hi = fmax(hi, dv[k]); }
  }
  lo = bminmax<NT>(lo, false, sh);
  hi = bminmax<NT>(hi, true, sh);
  int cnt = 0;
  unsigned keep = 0;
#pragma unroll
  for (int k = 0; k < kPer; ++k) {
    const int t = tid * kPer + k;
    if (t < T && (t == 0 || dv[k] >= double(tau))) { keep |= 1u << k; ++cnt; }
  }
  int L = 0;
  int pos = bscan_excl<NT>(cnt, L, sh);
#pragma unroll
  for (int k = 0; k < kPer; ++k) {
    if (keep & (1u << k)) {
      const int t = tid * kPer + k;
      sh.idx[pos] = t;
      sh.a[0][pos] = double(rel[t]);
      sh.g[0][pos] = hi > lo ? (dv[k] - lo) / (hi - lo) : 0.0;
      ++pos;
    }
  }
  __syncthreads();

  // ---- WTA: J-level gated Haar analysis (Eq. (9)-(10)) ------------------------
  int len = L, doff = 0, cur = 0;
  for (int lev = 0; lev < levels; ++lev) {
    const int half = (len + 1) / 2;
    if (tid == 0) { sh.lens[lev] = len; sh.doffs[lev] = doff; }
    const double* A0 = sh.a[cur];
    const double* G0 = sh.g[cur];
    for (int k = tid; k < half; k += NT) {
      const int i0 = 2 * k, i1 = min(2 * k + 1, len - 1);
      const double x0 = A0[i0], x1 = A0[i1];
      const double gp = 0.5 * (G0[i0] + G0[i1]);
      sh.a[cur ^ 1][k] = (x0 + x1) * inv_sqrt2;
      sh.g[cur ^ 1][k] = gp;
      sh.det[doff + k] = gp * ((x0 - x1) * inv_sqrt2);
    }
    __syncthreads();
    cur ^= 1;
    doff += half;
    len = half;
  }
  // ---- inverse DWT (Eq. (11)) ---------------------------------------------------
  for (int lev = levels - 1; lev >= 0; --lev) {
    const int plen = sh.lens[lev];
    const int half = (plen + 1) / 2;
    const double* A0 = sh.a[cur];
    double* A1 = sh.a[cur ^ 1];
    for (int k = tid; k < half; k += NT) {
      const double A = A0[k], D = sh.det[sh.doffs[lev] + k];
      A1[2 * k] = (A + D) * inv_sqrt2;
      if (2 * k + 1 < plen) A1[2 * k + 1] = (A - D) * inv_sqrt2;
    }
    __syncthreads();
    cur ^= 1;
  }
  const double* rt = sh.a[cur];  // r~ over the retained positions
  double* w = sh.g[cur ^ 1];      // free buffer: weights, then fractional parts

  // ---- budgets (Eq. (16), Eq. (5)) ------------------------------------------------
  const long long cap_total = (long long)L * N;
  if (B >= cap_total) {
    for (int i = tid; i < L; i += NT) sh.n[i] = N;
  } else {
    double wsum = 0.0;
    for (int i = tid; i < L; i += NT) {
      const double wi = fmax(rt[i], 0.0);
      w[i] = wi;
      wsum += wi;
    }
    wsum = bsum<NT>(wsum, sh);
    for (int i = tid; i < L; i += NT) {
      if (wsum == 0.0) w[i] = 1.0;
      sh.state[i] = w[i] > 0.0 ? kActive : kIdle;
      sh.n[i] = 0;
    }
    __syncthreads();
    long long R = B;
    while (R > 0) {
      int na = 0;
      for (int i = tid; i < L; i += NT) na += sh.state[i] == kActive;
      na = bsum_int<NT>(na, sh);
      if (na == 0) {  // every weighted frame is full: spread the rest evenly
        for (int i = tid; i < L; i += NT)
          if (sh.state[i] != kFull) { sh.state[i] = kActive; w[i] = 1.0; }
        __syncthreads();
      }
      double S = 0.0;
      for (int i = tid; i < L; i += NT)
        if (sh.state[i] == kActive) S += w[i];
      S = bsum<NT>(S, sh);
      const double Rd = double(R);
      int full = 0;
      for (int i = tid; i < L; i += NT)
        if (sh.state[i] == kActive && Rd * w[i] / S >= double(N)) ++full;
      full = bsum_int<NT>(full, sh);
      if (full > 0) {
        for (int i = tid; i < L; i += NT)
          if (sh.state[i] == kActive && Rd * w[i] / S >= double(N)) { sh.state[i] = kFull; sh.n[i] = N; }
        __syncthreads();
        R -= (long long)full * N;
        continue;
      }
      int base_sum = 0;
      for (int i = tid; i < L; i += NT) {
        if (sh.state[i] == kActive) {
          const double q = Rd * w[i] / S;
          const double b = floor(q);
          sh.n[i] = int(b);
          base_sum += int(b);
          w[i] = q - b;  // fractional part from here on
        }
      }
      const int left = int(R) - bsum_int<NT>(base_sum, sh);
      // +1 for the `left` active frames ranked first by (fraction desc, index asc)
      for (int i = tid; i < L; i += NT) {
        if (sh.state[i] != kActive) continue;
        const double f = w[i];
        int rank = 0;
        for (int j = 0; j < L; ++j) {
          if (sh.state[j] != kActive) continue;
          const double fj = w[j];
          rank += (fj > f) || (fj == f && j < i);
        }
        if (rank < left) sh.n[i] += 1;
      }
      R = 0;
    }
  }
  __syncthreads();

  // ---- scatter to frames, offsets, rectified relevance ----------------------------
  double* rr = w;  // per-frame r~ (weights no longer needed)
  for (int t = tid; t < T; t += NT) { sh.fb[t] = 0; rr[t] = 0.0; }
  __syncthreads();
  for (int i = tid; i < L; i += NT) {
    const int t = sh.idx[i];
    sh.fb[t] = sh.n[i];
    rr[t] = rt[i];
  }
  __syncthreads();
  for (int t = tid; t < T; t += NT) {
    budget[t] = sh.fb[t];
    if (rel_rect) rel_rect[t] = float(rr[t]);
  }
  int tsum = 0;
#pragma unroll
  for (int k = 0; k < kPer; ++k) {
    const int t = tid * kPer + k;
    tsum += t < T ? sh.fb[t] : 0;
  }
  int total = 0;
  int run = bscan_excl<NT>(tsum, total, sh);
#pragma unroll
  for (int k = 0; k < kPer; ++k) {
    const int t = tid * kPer + k;
    if (t < T) offset[t] = run;
    if (t < T) run += sh.fb[t];
  }
  if (tid == 0) offset[T] = total;
}

}  // namespace

hipError_t launch_temporal_budget(const wz_config& c, const float* frame_rel, const float* frame_delta,
                                  int32_t* budget, int32_t* offset, float* rel_rect, hipStream_t s) {
  const int N = c.H * c.W;
  if (c.T <= 64)
    hipLaunchKernelGGL((k_temporal_budget<64, 64>), dim3(1), dim3(64), 0, s, frame_rel, frame_delta, c.T, N,
                       (long long)c.B, c.levels, c.tau, budget, offset, rel_rect);
  else if (c.T <= 256)
    hipLaunchKernelGGL((k_temporal_budget<256, 256>), dim3(1), dim3(256), 0, s, frame_rel, frame_delta, c.T, N,
                       (long long)c.B, c.levels, c.tau, budget, offset, rel_rect);
  else
    hipLaunchKernelGGL((k_temporal_budget<1024, kTMax>), dim3(1), dim3(1024), 0, s, frame_rel, frame_delta, c.T, N,
                       (long long)c.B, c.levels, c.tau, budget, offset, rel_rect);
  return hipGetLastError();
}

}  // namespace wz
