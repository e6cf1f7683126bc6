// Stage 2: Wavelet Temporal Allocator (Sec. 3.2.2 gate and frame filter,
// Eq. (9)-(11)) and the integer frame budgets (Eq. (16) under Eq. (5)).
//
// The whole stage is a few hundred fp64 operations per frame, so it runs as
// ONE workgroup of 1024 threads with every array in LDS; frame t is handled by
// thread t (and t + 1024).  Steps:
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

constexpr int kThreads = 1024;
constexpr int kWaves = kThreads / kWave;
constexpr int kTMax = 2048;
constexpr int kPer = kTMax / kThreads;  // frames per thread
constexpr int kMaxLevels = 16;

enum : unsigned char { kIdle = 0, kActive = 1, kFull = 2 };

struct Shared {
  double a[kTMax];                  // approximation being transformed, then r~
  double g[kTMax];                  // gate, pooled with the approximation
  double det[kTMax + kMaxLevels];   // gated detail coefficients of every level
  double w[kTMax];                  // weights, then fractional parts
  int idx[kTMax];                   // frame index of each retained position
  int n[kTMax];                     // budget of each retained position
  int fb[kTMax];                    // budget of each frame
  unsigned char state[kTMax];
  double dred[kWaves];
  int ired[kWaves];
  int lens[kMaxLevels];
  int doffs[kMaxLevels];
};

__device__ double block_sum(double v, Shared& sh) {
  v = wave_sum_f64(v);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) sh.dred[wave] = v;
  __syncthreads();
  double s = 0.0;
#pragma unroll
  for (int i = 0; i < kWaves; ++i) s += sh.dred[i];
  return s;
}

__device__ double block_min_max(double v, bool want_max, Shared& sh) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) {
    const double o = __shfl_xor(v, m, kWave);
    v = want_max ? fmax(v, o) : fmin(v, o);
  }
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) sh.dred[wave] = v;
  __syncthreads();
  double r = sh.dred[0];
  for (int i = 1; i < kWaves; ++i) r = want_max ? fmax(r, sh.dred[i]) : fmin(r, sh.dred[i]);
  return r;
}

__device__ int block_sum_int(int v, Shared& sh) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, kWave);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) sh.ired[wave] = v;
  __syncthreads();
  int s = 0;
#pragma unroll
  for (int i = 0; i < kWaves; ++i) s += sh.ired[i];
  return s;
}

// Exclusive prefix sum of v over the block in thread order (thread i's
// contribution precedes thread i+1's); returns the prefix, `total` gets the sum.
__device__ int block_exclusive_scan(int v, int& total, Shared& sh) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int inc = v;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const int o = __shfl_up(inc, d, kWave);
    if (lane >= d) inc += o;
  }
  __syncthreads();
  if (lane == 63) sh.ired[wave] = inc;
  __syncthreads();
  int before = 0;
  total = 0;
  for (int i = 0; i < kWaves; ++i) {
    if (i < wave) before += sh.ired[i];
    total += sh.ired[i];
  }
  return before + inc - v;
}

__global__ __launch_bounds__(kThreads) void k_temporal_budget(const float* __restrict__ rel,
                                                              const float* __restrict__ delta, int T, int N,
                                                              long long B, int levels, float tau,
                                                              int32_t* __restrict__ budget,
                                                              int32_t* __restrict__ offset,
                                                              float* __restrict__ rel_rect) {
  __shared__ Shared sh;
  const int tid = threadIdx.x;
  const double inv_sqrt2 = 0.70710678118654752440;

  // ---- gamma = min-max(delta); retained set M --------------------------------
  double dv[kPer], lo = INFINITY, hi = -INFINITY;
#pragma unroll
  for (int k = 0; k < kPer; ++k) {
    const int t = tid * kPer + k;
    dv[k] = t < T ? double(delta[t]) : 0.0;
    if (t < T) { lo = fmin(lo, dv[k]); hi = fmax(hi, dv[k]); }
  }
  lo = block_min_max(lo, false, sh);
  hi = block_min_max(hi, true, sh);
  int keep[kPer], cnt = 0;
#pragma unroll
  for (int k = 0; k < kPer; ++k) {
    const int t = tid * kPer + k;
    keep[k] = t < T && (t == 0 || dv[k] >= double(tau));
    cnt += keep[k];
  }
  int L = 0;
  int pos = block_exclusive_scan(cnt, L, sh);
#pragma unroll
  for (int k = 0; k < kPer; ++k) {
    const int t = tid * kPer + k;
    if (keep[k]) {
      sh.idx[pos] = t;
      sh.a[pos] = double(rel[t]);
      sh.g[pos] = hi > lo ? (dv[k] - lo) / (hi - lo) : 0.0;
      ++pos;
    }
  }
  __syncthreads();

  // ---- WTA: J-level gated Haar analysis ---------------------------------------
  int len = L, doff = 0;
  for (int lev = 0; lev < levels; ++lev) {
    const int half = (len + 1) / 2;  // <= kThreads because L <= kTMax
    if (tid == 0) { sh.lens[lev] = len; sh.doffs[lev] = doff; }
    double A = 0.0, Dg = 0.0, gp = 0.0;
    if (tid < half) {
      const int i0 = 2 * tid, i1 = min(2 * tid + 1, len - 1);
      const double x0 = sh.a[i0], x1 = sh.a[i1];
      A = (x0 + x1) * inv_sqrt2;
      const double D = (x0 - x1) * inv_sqrt2;
      gp = 0.5 * (sh.g[i0] + sh.g[i1]);
      Dg = gp * D;
    }
    __syncthreads();
    if (tid < half) { sh.a[tid] = A; sh.g[tid] = gp; sh.det[doff + tid] = Dg; }
    __syncthreads();
    doff += half;
    len = half;
  }
  // ---- inverse DWT (Eq. (11)) --------------------------------------------------
  for (int lev = levels - 1; lev >= 0; --lev) {
    const int plen = sh.lens[lev];
    const int half = (plen + 1) / 2;
    double e = 0.0, o = 0.0;
    if (tid < half) {
      const double A = sh.a[tid], D = sh.det[sh.doffs[lev] + tid];
      e = (A + D) * inv_sqrt2;
      o = (A - D) * inv_sqrt2;
    }
    __syncthreads();
    if (tid < half) {
      sh.a[2 * tid] = e;
      if (2 * tid + 1 < plen) sh.a[2 * tid + 1] = o;
    }
    __syncthreads();
  }

  // ---- budgets (Eq. (16), Eq. (5)) ----------------------------------------------
  const long long cap_total = (long long)L * N;
  if (B >= cap_total) {
    for (int i = tid; i < L; i += kThreads) sh.n[i] = N;
  } else {
    double wsum = 0.0;
    for (int i = tid; i < L; i += kThreads) {
      const double w = fmax(sh.a[i], 0.0);
      sh.w[i] = w;
      wsum += w;
    }
    wsum = block_sum(wsum, sh);
    for (int i = tid; i < L; i += kThreads) {
      if (wsum == 0.0) sh.w[i] = 1.0;
      sh.state[i] = sh.w[i] > 0.0 ? kActive : kIdle;
      sh.n[i] = 0;
    }
    __syncthreads();
    long long R = B;
    while (R > 0) {
      int na = 0;
      for (int i = tid; i < L; i += kThreads) na += sh.state[i] == kActive;
      na = block_sum_int(na, sh);
      if (na == 0) {  // every weighted frame is full: spread the rest evenly
        for (int i = tid; i < L; i += kThreads)
          if (sh.state[i] != kFull) { sh.state[i] = kActive; sh.w[i] = 1.0; }
        __syncthreads();
      }
      double S = 0.0;
      for (int i = tid; i < L; i += kThreads)
        if (sh.state[i] == kActive) S += sh.w[i];
      S = block_sum(S, sh);
      const double Rd = double(R);
      int full = 0;
      for (int i = tid; i < L; i += kThreads)
        if (sh.state[i] == kActive && Rd * sh.w[i] / S >= double(N)) ++full;
      full = block_sum_int(full, sh);
      if (full > 0) {
        for (int i = tid; i < L; i += kThreads)
          if (sh.state[i] == kActive && Rd * sh.w[i] / S >= double(N)) { sh.state[i] = kFull; sh.n[i] = N; }
        __syncthreads();
        R -= (long long)full * N;
        continue;
      }
      int base_sum = 0;
      for (int i = tid; i < L; i += kThreads) {
        if (sh.state[i] == kActive) {
          const double q = Rd * sh.w[i] / S;
          const double b = floor(q);
          sh.n[i] = int(b);
          base_sum += int(b);
          sh.w[i] = q - b;  // fractional part from here on
        }
      }
      const int left = int(R) - block_sum_int(base_sum, sh);
      // rank of each active frame by (fraction desc, index asc)
      int plus[kPer];
#pragma unroll
      for (int k = 0; k < kPer; ++k) {
        const int i = tid + k * kThreads;
        plus[k] = 0;
        if (i < L && sh.state[i] == kActive) {
          const double f = sh.w[i];
          int rank = 0;
          for (int j = 0; j < L; ++j) {
            if (sh.state[j] != kActive) continue;
            const double fj = sh.w[j];
            rank += (fj > f) || (fj == f && j < i);
          }
          plus[k] = rank < left;
        }
      }
      __syncthreads();
#pragma unroll
      for (int k = 0; k < kPer; ++k) {
        const int i = tid + k * kThreads;
        if (i < L) sh.n[i] += plus[k];
      }
      R = 0;
    }
  }
  __syncthreads();

  // ---- scatter to frames, offsets, rectified relevance ----------------------------
  for (int t = tid; t < T; t += kThreads) { sh.fb[t] = 0; sh.g[t] = 0.0; }
  __syncthreads();
  for (int i = tid; i < L; i += kThreads) {
    const int t = sh.idx[i];
    sh.fb[t] = sh.n[i];
    sh.g[t] = sh.a[i];
  }
  __syncthreads();
  for (int t = tid; t < T; t += kThreads) {
    budget[t] = sh.fb[t];
    if (rel_rect) rel_rect[t] = float(sh.g[t]);
  }
  int nv[kPer], tsum = 0;
#pragma unroll
  for (int k = 0; k < kPer; ++k) {
    const int t = tid * kPer + k;
    nv[k] = t < T ? sh.fb[t] : 0;
    tsum += nv[k];
  }
  int total = 0;
  int run = block_exclusive_scan(tsum, total, sh);
#pragma unroll
  for (int k = 0; k < kPer; ++k) {
    const int t = tid * kPer + k;
    if (t < T) offset[t] = run;
    run += nv[k];
  }
  if (tid == 0) offset[T] = total;
}

}  // namespace

hipError_t launch_temporal_budget(const wz_config& c, const float* frame_rel, const float* frame_delta,
                                  int32_t* budget, int32_t* offset, float* rel_rect, hipStream_t s) {
  hipLaunchKernelGGL(k_temporal_budget, dim3(1), dim3(kThreads), 0, s, frame_rel, frame_delta, c.T,
                     c.H * c.W, (long long)c.B, c.levels, c.tau, budget, offset, rel_rect);
  return hipGetLastError();
}

}  // namespace wz
