// Integer frame budgets of the Wavelet Temporal Allocator (gate and frame
// filter of Sec. 3.2.2; Sec. 3.2.3, Eq. (9)-(11)) under Eq. (16) and Eq. (5)
// (Sec. 3.2.4), as device code
// run by ONE workgroup (or one wave) from r_t and delta_t.  Included by the
// standalone budget kernel and by the fused selection and gather kernel.
//
// The budget is a few fp64 operations per frame, so it runs in ONE workgroup
// with every array in LDS, or in one wave: up to T = 64 with every value in
// registers (budget_wave_compute), up to T = 256 with four frames per lane,
// also in registers (budget_wave_slots; budget_body with NT = 64 keeps the
// same layout in LDS, for the filter-bank bases); 1024 threads beyond.
// Steps:
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
//   (db4 / bior4.4 temporal bases: the same steps with the filter bank of
//   wz_wavelets.h, the gate pooled to each level's detail length by adaptive
//   average pooling; workgroup version only)
#pragma once

#include "wz_device.h"
#include "wz_wavelets.h"

namespace wz {
namespace {

constexpr int kTMax = kMaxFrames;
constexpr int kMaxLevels = 16;

enum : unsigned char { kIdle = 0, kActive = 1, kFull = 2 };

template <int TV>
struct Shared {
  double a[2][TV];              // approximation (ping-pong), then r~ in a[0]
  double g[2][TV];              // gate pooled alongside (ping-pong); g[0] reused for weights
  double det[TV + 8 * kMaxLevels];  // gated detail coefficients of every level
  int idx[TV];                  // frame index of each retained position
  int n[TV];                    // budget of each retained position
  int fb[TV];                   // budget of each frame
  unsigned char state[TV];
  double dred[16];
  int ired[16];
  int lens[kMaxLevels];
  int doffs[kMaxLevels];
};

// Block-wide ordering point of the budget body: a barrier for several waves;
// one wave only needs its LDS accesses kept in program order.
template <int NT>
__device__ __forceinline__ void bsync() {
  if constexpr (NT > kWave) {
    __syncthreads();
  } else {
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    __builtin_amdgcn_wave_barrier();
  }
}

template <int NT, typename Sh>
__device__ double bsum(double v, Sh& sh) {
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

template <int NT, typename Sh>
__device__ double bminmax(double v, bool want_max, Sh& sh) {
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

template <int NT, typename Sh>
__device__ int bsum_int(int v, Sh& sh) {
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
template <int NT, typename Sh>
__device__ int bscan_excl(int v, int& total, Sh& sh) {
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

// One wave hands the `need` extra tokens of the last apportionment round to
// the active positions ranked first by (fractional part desc, index asc);
// position i is lane i % 64's slot i / 64, its fractional part in w[i].
// Non-negative doubles order like their bit patterns, so a descent over the
// bits finds them: positions with the current bit set are taken whole while
// they fit, else the search continues among them; positions still tied after
// the last bit go by index (slot, then lane).
template <int TV, typename Sh>
__device__ void remainder_extras_wave(const double* w, Sh& sh, int L, int need) {
  constexpr int SL = (TV + kWave - 1) / kWave;
  const int lane = threadIdx.x & 63;
  uint64_t fb[SL], cand[SL], chosen[SL];
  uint64_t any = 0ull, all = ~0ull;
#pragma unroll
  for (int s = 0; s < SL; ++s) {
    const int i = s * kWave + lane;
    const bool act = i < L && sh.state[i] == kActive;
    fb[s] = act ? __builtin_bit_cast(uint64_t, w[i]) : 0ull;
    cand[s] = __ballot(act);
    chosen[s] = 0ull;
    if (act) {
      any |= fb[s];
      all &= fb[s];
    }
  }
  // bits on which every active position agrees decide nothing: start below them
  any = wave_reduce_u64(any, [](uint64_t x, uint64_t y) { return x | y; });
  all = wave_reduce_u64(all, [](uint64_t x, uint64_t y) { return x & y; });
  const int top = (any ^ all) ? 63 - __clzll(any ^ all) : -1;
  for (int bit = top; bit >= 0 && need > 0; --bit) {
    int cnt = 0;
#pragma unroll
    for (int s = 0; s < SL; ++s) cnt += __popcll(cand[s]);
    if (cnt <= need) break;
    uint64_t ones[SL];
    int c1 = 0;
#pragma unroll
    for (int s = 0; s < SL; ++s) {
      ones[s] = cand[s] & __ballot((fb[s] >> bit) & 1ull);
      c1 += __popcll(ones[s]);
    }
    if (c1 <= need) {
#pragma unroll
      for (int s = 0; s < SL; ++s) {
        chosen[s] |= ones[s];
        cand[s] &= ~ones[s];
      }
      need -= c1;
    } else {
#pragma unroll
      for (int s = 0; s < SL; ++s) cand[s] = ones[s];
    }
  }
  // the remaining candidates all fit, or are exact ties: smaller index first
#pragma unroll
  for (int s = 0; s < SL; ++s)
    for (; need > 0 && cand[s]; --need) {
      chosen[s] |= cand[s] & (~cand[s] + 1ull);
      cand[s] &= cand[s] - 1ull;
    }
#pragma unroll
  for (int s = 0; s < SL; ++s) {
    const int i = s * kWave + lane;
    if (i < L && ((chosen[s] >> lane) & 1ull)) sh.n[i] += 1;
  }
}

// NT threads handle up to TV frames; thread tid owns frames tid*kPer .. tid*kPer+kPer-1.
// bank: the temporal filter bank (null: Haar).
template <int NT, int TV>
__device__ void budget_body(const float* __restrict__ rel, const float* __restrict__ delta, int T, int N,
                            long long B, int levels, float tau, int32_t* __restrict__ budget,
                            int32_t* __restrict__ offset, float* __restrict__ rel_rect,
                            const Bank* bank_in = nullptr) {
  constexpr int kPer = (TV + NT - 1) / NT;  // frames per thread (contiguous run)
  static_assert(kPer <= 32 && TV <= kTMax, "frame mask holds 32 frames per thread");
  __shared__ Shared<TV> sh;
  const int tid = threadIdx.x;
  const double inv_sqrt2 = 0.70710678118654752440;

  // ---- gamma = min-max(delta); retained set M (thread tid owns frames tid*kPer ..) ----
  double dv[kPer], rv[kPer], lo = INFINITY, hi = -INFINITY;
#pragma unroll
  for (int k = 0; k < kPer; ++k) {
    const int t = tid * kPer + k;
    dv[k] = t < T ? double(delta[t]) : 0.0;
    rv[k] = t < T ? double(rel[t]) : 0.0;
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
      sh.a[0][pos] = rv[k];
      sh.g[0][pos] = hi > lo ? (dv[k] - lo) / (hi - lo) : 0.0;
      ++pos;
    }
  }
  bsync<NT>();

  int len = L, doff = 0, cur = 0;
  if (bank_in) {
    // ---- WTA with a filter bank: analysis, gate pooled to the detail length,
    // gated details (Eq. (9)-(10)); every level's coefficients stay within TV
    // entries (n <= max(len, 8) for F <= 10); the taps are read from LDS ----
    __shared__ Bank s_bank;
    if (tid == 0) s_bank = *bank_in;
    bsync<NT>();
    const Bank* bank = &s_bank;
    const int F = bank->F;
    for (int lev = 0; lev < levels; ++lev) {
      const int n = bank_len(len, F);
      if (tid == 0) { sh.lens[lev] = len; sh.doffs[lev] = doff; }
      const double* A0 = sh.a[cur];
      const double* G0 = sh.g[cur];
      for (int k = tid; k < n; k += NT) {
        double a = 0.0, d = 0.0;
        for (int j = 0; j < F; ++j) {
          const double x = A0[sym_index(2 * k + 1 - j, len)];
          a += bank->dec_lo[j] * x;
          d += bank->dec_hi[j] * x;
        }
        // gate: the mean of G0 over inputs floor(k len / n) .. ceil((k + 1) len / n) - 1
        const int lo = (k * len) / n, hi = ((k + 1) * len + n - 1) / n;
        double gs = 0.0;
        for (int i = lo; i < hi; ++i) gs += G0[i];
        const double gp = gs / double(hi - lo);
        sh.a[cur ^ 1][k] = a;
        sh.g[cur ^ 1][k] = gp;
        sh.det[doff + k] = gp * d;
      }
      bsync<NT>();
      cur ^= 1;
      doff += n;
      len = n;
    }
    // ---- inverse (Eq. (11)): each level rebuilt and cropped to its length ----
    for (int lev = levels - 1; lev >= 0; --lev) {
      const int plen = sh.lens[lev], n = bank_len(plen, F);
      const double* A0 = sh.a[cur];
      const double* D0 = sh.det + sh.doffs[lev];
      double* A1 = sh.a[cur ^ 1];
      for (int i = tid; i < plen; i += NT) {
        double s = 0.0;
        for (int k = max(0, (i - 1) / 2); k < n; ++k) {  // rec index i + F - 2 - 2k in [0, F)
          const int f = i + F - 2 - 2 * k;
          if (f < 0) break;
          if (f < F) s += bank->rec_lo[f] * A0[k] + bank->rec_hi[f] * D0[k];
        }
        A1[i] = s;
      }
      bsync<NT>();
      cur ^= 1;
    }
  } else {
  // ---- WTA: J-level gated Haar analysis (Eq. (9)-(10)) ------------------------
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
    bsync<NT>();
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
    bsync<NT>();
    cur ^= 1;
  }
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
    bsync<NT>();
    long long R = B;
    while (R > 0) {
      int na = 0;
      for (int i = tid; i < L; i += NT) na += sh.state[i] == kActive;
      na = bsum_int<NT>(na, sh);
      if (na == 0) {  // every weighted frame is full: spread the rest evenly
        for (int i = tid; i < L; i += NT)
          if (sh.state[i] != kFull) { sh.state[i] = kActive; w[i] = 1.0; }
        bsync<NT>();
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
        bsync<NT>();
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
          w[i] = q - b;  // fractional part from here on (in [0, 1))
        } else {
          w[i] = -1.0;  // below every fractional part: never ranks ahead
        }
      }
      const int left = int(R) - bsum_int<NT>(base_sum, sh);
      // +1 for the `left` active frames ranked first by (fraction desc, index asc)
      if constexpr (NT == kWave) {
        bsync<NT>();
        remainder_extras_wave<TV>(w, sh, L, left);
      } else
      for (int i = tid; i < L; i += NT) {
        if (sh.state[i] != kActive) continue;
        const double f = w[i];
        // branch-free counting, eight loads in flight at a time
        int rank = 0, j = 0;
        for (; j + 8 <= L; j += 8) {
          double fj[8];
#pragma unroll
          for (int e = 0; e < 8; ++e) fj[e] = w[j + e];
#pragma unroll
          for (int e = 0; e < 8; ++e) rank += int(fj[e] > f) | (int(fj[e] == f) & int(j + e < i));
        }
        for (; j < L; ++j) {
          const double fj = w[j];
          rank += int(fj > f) | (int(fj == f) & int(j < i));
        }
        if (rank < left) sh.n[i] += 1;
      }
      R = 0;
    }
  }
  bsync<NT>();

  // ---- scatter to frames, offsets, rectified relevance ----------------------------
  double* rr = w;  // per-frame r~ (weights no longer needed)
  for (int t = tid; t < T; t += NT) { sh.fb[t] = 0; rr[t] = 0.0; }
  bsync<NT>();
  for (int i = tid; i < L; i += NT) {
    const int t = sh.idx[i];
    sh.fb[t] = sh.n[i];
    rr[t] = rt[i];
  }
  bsync<NT>();
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


// ---------------------------------------------------------------------------
// T <= 64: one wave, frame t (then retained position i) in lane t (lane i),
// every value in registers.  Reductions use DPP row permutations and lane
// reads instead of LDS round trips; compaction uses a ballot; the Haar levels
// move data with lane shuffles.  Same arithmetic as budget_body.
// ---------------------------------------------------------------------------
// Runs on one whole wave (wave 0 of its workgroup).  Lane t holds delta_t
// and r_t (anything for lanes >= T); outputs may point to global memory or
// LDS; det is LDS for every level's detail coefficients, [levels][kWave].
__device__ __forceinline__ void budget_wave_compute_det(double d, double r, int T, int N, long long B, int levels,
                                                        float tau, int32_t* __restrict__ budget,
                                                        int32_t* __restrict__ offset, float* __restrict__ rel_rect,
                                                        double* __restrict__ det) {
  const double inv_sqrt2 = 0.70710678118654752440;
  auto dadd = [](double a, double b) { return a + b; };
  const int lane = threadIdx.x & 63;
  const bool valid = lane < T;

  // ---- gamma = min-max(delta); retained set M in temporal order ----
  // delta arrives in fp32, so its extremes are exact in fp32
  const double lo = double(wave_min_f32(valid ? float(d) : INFINITY));
  const double hi = double(wave_max_f32(valid ? float(d) : -INFINITY));
  const double gam = hi > lo ? (d - lo) / (hi - lo) : 0.0;
  const bool keep = valid && (lane == 0 || d >= double(tau));
  const uint64_t kmask = __ballot(keep);
  const int L = __popcll(kmask);
  const int pos = __popcll(kmask & ((1ull << lane) - 1ull));
  // a permutation of the lanes: retained frames to positions 0..L-1, the rest after them
  const int dst = keep ? pos : L + (lane - pos);
  double x = permute_f64(dst, r);  // position i: r of the i-th retained frame
  double g = permute_f64(dst, gam);

  // ---- WTA: J-level gated Haar analysis (Eq. (9)-(10)); lanes beyond a
  // level's length hold values nobody reads ----
  int len = L;
  for (int lev = 0; lev < levels; ++lev) {
    const int i0 = min(2 * lane, kWave - 1), i1 = min(min(2 * lane + 1, len - 1), kWave - 1);
    const double x0 = __shfl(x, i0, kWave), x1 = __shfl(x, i1, kWave);
    const double gp = 0.5 * (__shfl(g, i0, kWave) + __shfl(g, i1, kWave));
    det[lev * kWave + lane] = gp * ((x0 - x1) * inv_sqrt2);
    x = (x0 + x1) * inv_sqrt2;
    g = gp;
    len = (len + 1) / 2;
  }
  // ---- inverse DWT (Eq. (11)) ----
  for (int lev = levels - 1; lev >= 0; --lev) {
    const int k = lane >> 1;
    const double A = __shfl(x, k, kWave), Dk = det[lev * kWave + k];
    x = (lane & 1) ? (A - Dk) * inv_sqrt2 : (A + Dk) * inv_sqrt2;
  }
  // x in lane i < L: r~ of retained position i

  // ---- budgets (Eq. (16), Eq. (5)) ----
  const bool inM = lane < L;
  int n = 0;
  if (B >= (long long)L * N) {
    n = inM ? N : 0;
  } else {
    double w = inM ? fmax(x, 0.0) : 0.0;
    const double wsum = wave_reduce_f64(w, dadd);
    if (wsum == 0.0 && inM) w = 1.0;
    uint64_t active = __ballot(inM && w > 0.0), full = 0;
    long long R = B;
    while (R > 0) {
      if (active == 0) {  // every weighted frame is full: spread the rest evenly
        active = __ballot(inM) & ~full;
        if ((active >> lane) & 1) w = 1.0;
      }
      const bool act = (active >> lane) & 1;
      const double S = wave_reduce_f64(act ? w : 0.0, dadd);
      const double Rd = double(R);
      const double q = act ? Rd * w / S : 0.0;
      const uint64_t cap = __ballot(act && q >= double(N));
      if (cap) {
        if ((cap >> lane) & 1) n = N;
        full |= cap;
        active &= ~cap;
        R -= (long long)__popcll(cap) * N;
        continue;
      }
      const double b = floor(q);
      if (act) n = int(b);
      const double frac = act ? q - b : 0.0;  // in [0, 1) for active positions
      int need = int(R) - wave_reduce_sum_i32(act ? int(b) : 0);
      // +1 for the `need` active positions ranked first by (fraction desc,
      // index asc).  Non-negative doubles order like their bit patterns, so a
      // descent over the bits (fractions below 1 leave bits 63 and 62 clear)
      // finds them: positions with the current bit set are taken whole while
      // they fit, else the search continues among them; positions still tied
      // after the last bit go by index.
      const uint64_t fb = __builtin_bit_cast(uint64_t, frac);
      // bits on which every active position agrees decide nothing: start
      // below them
      const uint64_t any = wave_reduce_u64(act ? fb : 0ull, [](uint64_t x, uint64_t y) { return x | y; });
      const uint64_t all = wave_reduce_u64(act ? fb : ~0ull, [](uint64_t x, uint64_t y) { return x & y; });
      const int top = (any ^ all) ? 63 - __clzll(any ^ all) : -1;
      uint64_t cand = active, chosen = 0;
      for (int bit = top; bit >= 0 && need > 0; --bit) {
        if (int(__popcll(cand)) <= need) break;
        const uint64_t ones = cand & __ballot((fb >> bit) & 1ull);
        const int c1 = __popcll(ones);
        if (c1 <= need) {
          chosen |= ones;
          need -= c1;
          cand &= ~ones;
        } else {
          cand = ones;
        }
      }
      for (; need > 0 && cand; --need) {  // the remaining candidates all fit, or are exact ties
        chosen |= cand & (~cand + 1ull);
        cand &= cand - 1ull;
      }
      if ((chosen >> lane) & 1ull) n += 1;
      R = 0;
    }
  }

  // ---- back to frames, offsets, rectified relevance ----
  const int nb = __shfl(n, pos, kWave);
  const double rt = __shfl(x, pos, kWave);
  const int bt = keep ? nb : 0;
  const int incl = wave_incl_scan_i32(bt);
  if (valid) {
    budget[lane] = bt;
    offset[lane] = incl - bt;
    if (rel_rect) rel_rect[lane] = keep ? float(rt) : 0.f;
  }
  if (lane == T - 1) offset[T] = incl;
}
// The same with the detail coefficients in a static LDS array of its own.
__device__ void budget_wave_compute(double d, double r, int T, int N, long long B, int levels, float tau,
                                    int32_t* __restrict__ budget, int32_t* __restrict__ offset,
                                    float* __restrict__ rel_rect) {
  __shared__ double s_det[kMaxLevels * kWave];
  budget_wave_compute_det(d, r, T, N, B, levels, tau, budget, offset, rel_rect, s_det);
}

// ---------------------------------------------------------------------------
// T <= TV (TV = 64 SL, at most 256): one wave, frame t and retained position
// i in slot t / 64 (i / 64) of lane t % 64 (i % 64), every value in
// registers except each level's detail coefficients (LDS); the compaction
// to the retained positions and the way back go through LDS only when the
// frame filter drops a frame.  The positions' layout is budget_body<64, TV>'s
// and so are its sums (a lane's slots in order, then the same butterfly), so
// the budgets are bit for bit that function's; its LDS arrays and their
// ordering points are what this version saves.
// ---------------------------------------------------------------------------
template <int TV>
__device__ void budget_wave_slots(const float* __restrict__ rel, const float* __restrict__ delta, int T, int N,
                                  long long B, int levels, float tau, int32_t* __restrict__ budget,
                                  int32_t* __restrict__ offset, float* __restrict__ rel_rect) {
  constexpr int SL = TV / kWave;
  static_assert(TV % kWave == 0 && SL >= 1 && SL <= 4, "one to four slots per lane");
  const double inv_sqrt2 = 0.70710678118654752440;
  const int lane = threadIdx.x & 63;
  const uint64_t below = (1ull << lane) - 1ull;  // lanes before this one
  __shared__ double s_det[TV + kMaxLevels];  // every level's gated details, level after level
  __shared__ int s_doff[kMaxLevels];        // where each level's start
  __shared__ double s_mv[2][TV];
  __shared__ int s_nmv[TV];
  auto order = []() {  // one wave: its LDS accesses in program order
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    __builtin_amdgcn_wave_barrier();
  };

  // ---- gamma = min-max(delta); retained set M ----
  double x[SL], g[SL];
  bool keep[SL];
  uint64_t kmask[SL];
  int kpos[SL];  // retained position of the slot's frame
  float dlo = INFINITY, dhi = -INFINITY;
  double dv[SL];
#pragma unroll
  for (int s = 0; s < SL; ++s) {
    const int t = s * kWave + lane;
    const bool valid = t < T;
    const float df = valid ? delta[t] : 0.f;
    dv[s] = double(df);
    x[s] = valid ? double(rel[t]) : 0.0;
    if (valid) {
      dlo = fminf(dlo, df);
      dhi = fmaxf(dhi, df);
    }
    keep[s] = valid && (t == 0 || dv[s] >= double(tau));
    kmask[s] = __ballot(keep[s]);
  }
  // delta arrives in fp32, so its extremes are exact in fp32
  const double lo = double(wave_min_f32(dlo)), hi = double(wave_max_f32(dhi));
  int L = 0;
#pragma unroll
  for (int s = 0; s < SL; ++s) {
    g[s] = hi > lo ? (dv[s] - lo) / (hi - lo) : 0.0;
    kpos[s] = L + __popcll(kmask[s] & below);
    L += __popcll(kmask[s]);
  }
  const bool moved = L < T;  // uniform: some frame dropped, positions differ from frames
  if (moved) {
#pragma unroll
    for (int s = 0; s < SL; ++s)
      if (keep[s]) {
        s_mv[0][kpos[s]] = x[s];
        s_mv[1][kpos[s]] = g[s];
      }
    order();
#pragma unroll
    for (int s = 0; s < SL; ++s) {
      x[s] = s_mv[0][s * kWave + lane];  // positions past L: values nobody reads
      g[s] = s_mv[1][s * kWave + lane];
    }
  }

  // ---- WTA: J-level gated Haar analysis (Eq. (9)-(10)); output k = 64 s +
  // lane reads inputs 2k and min(2k + 1, len - 1), both in slot 2s or 2s + 1
  int len = L, doff = 0;
  for (int lev = 0; lev < levels; ++lev) {
    const int half = (len + 1) / 2;
    if (lane == 0) s_doff[lev] = doff;
    double xn[SL], gn[SL];
#pragma unroll
    for (int s = 0; s < SL; ++s) {
      xn[s] = 0.0;
      gn[s] = 0.0;
      if constexpr (true) {
        const int k = s * kWave + lane;
        const int i0 = 2 * k, i1 = min(2 * k + 1, max(len - 1, 0));
        auto fetch = [&](const double (&v)[SL], int i) {
          // slot 2s or 2s + 1 (the value of a slot past the array is never used)
          const double a = 2 * s < SL ? __shfl(v[min(2 * s, SL - 1)], i & 63, kWave) : 0.0;
          const double b = 2 * s + 1 < SL ? __shfl(v[min(2 * s + 1, SL - 1)], i & 63, kWave) : 0.0;
          return (i >> 6) == 2 * s ? a : b;
        };
        if (2 * s < SL) {
          const double x0 = fetch(x, i0), x1 = fetch(x, i1);
          const double gp = 0.5 * (fetch(g, i0) + fetch(g, i1));
          if (k < half) s_det[doff + k] = gp * ((x0 - x1) * inv_sqrt2);
          xn[s] = (x0 + x1) * inv_sqrt2;
          gn[s] = gp;
        }
      }
    }
#pragma unroll
    for (int s = 0; s < SL; ++s) {
      x[s] = xn[s];
      g[s] = gn[s];
    }
    doff += half;
    len = half;
  }
  order();
  // ---- inverse DWT (Eq. (11)): output i = 64 s + lane from coefficient
  // k = i / 2 (slot s / 2, lane 32 (s % 2) + lane / 2) ----
  for (int lev = levels - 1; lev >= 0; --lev) {
    const int d0 = s_doff[lev];
    double xn[SL];
#pragma unroll
    for (int s = 0; s < SL; ++s) {
      const int i = s * kWave + lane, k = i >> 1;
      const double A = __shfl(x[s >> 1], 32 * (s & 1) + (lane >> 1), kWave);
      const double D = s_det[min(d0 + k, TV + kMaxLevels - 1)];  // past the level: a value nobody uses
      xn[s] = (i & 1) ? (A - D) * inv_sqrt2 : (A + D) * inv_sqrt2;
    }
#pragma unroll
    for (int s = 0; s < SL; ++s) x[s] = xn[s];
  }
  // x[s] at position 64 s + lane < L: r~ of that retained position

  // ---- budgets (Eq. (16), Eq. (5)) ----
  int n[SL];
  uint64_t inM[SL];
#pragma unroll
  for (int s = 0; s < SL; ++s) {
    n[s] = 0;
    inM[s] = __ballot(s * kWave + lane < L);
  }
  if (B >= (long long)L * N) {
#pragma unroll
    for (int s = 0; s < SL; ++s) n[s] = s * kWave + lane < L ? N : 0;
  } else {
    double w[SL], wsum = 0.0;
#pragma unroll
    for (int s = 0; s < SL; ++s) {
      w[s] = s * kWave + lane < L ? fmax(x[s], 0.0) : 0.0;
      if (s * kWave + lane < L) wsum += w[s];
    }
    wsum = wave_sum_f64(wsum);
    uint64_t active[SL], full[SL];
#pragma unroll
    for (int s = 0; s < SL; ++s) {
      if (wsum == 0.0 && s * kWave + lane < L) w[s] = 1.0;
      active[s] = __ballot(s * kWave + lane < L && w[s] > 0.0);
      full[s] = 0ull;
    }
    long long R = B;
    while (R > 0) {
      int na = 0;
#pragma unroll
      for (int s = 0; s < SL; ++s) na += __popcll(active[s]);
      if (na == 0) {  // every weighted frame is full: spread the rest evenly
#pragma unroll
        for (int s = 0; s < SL; ++s) {
          active[s] = inM[s] & ~full[s];
          if ((active[s] >> lane) & 1ull) w[s] = 1.0;
        }
      }
      double S = 0.0;
#pragma unroll
      for (int s = 0; s < SL; ++s)
        if ((active[s] >> lane) & 1ull) S += w[s];
      S = wave_sum_f64(S);
      const double Rd = double(R);
      double q[SL];
      int nfull = 0;
      uint64_t cap[SL];
#pragma unroll
      for (int s = 0; s < SL; ++s) {
        const bool act = (active[s] >> lane) & 1ull;
        q[s] = act ? Rd * w[s] / S : 0.0;
        cap[s] = __ballot(act && q[s] >= double(N));
        nfull += __popcll(cap[s]);
      }
      if (nfull > 0) {
#pragma unroll
        for (int s = 0; s < SL; ++s) {
          if ((cap[s] >> lane) & 1ull) n[s] = N;
          full[s] |= cap[s];
          active[s] &= ~cap[s];
        }
        R -= (long long)nfull * N;
        continue;
      }
      int base_sum = 0;
      uint64_t fb[SL], cand[SL], chosen[SL];
      uint64_t any = 0ull, all = ~0ull;
#pragma unroll
      for (int s = 0; s < SL; ++s) {
        const bool act = (active[s] >> lane) & 1ull;
        const double b = floor(q[s]);
        if (act) {
          n[s] = int(b);
          base_sum += int(b);
        }
        // fractional parts in [0, 1): non-negative doubles order like their
        // bit patterns
        fb[s] = act ? __builtin_bit_cast(uint64_t, q[s] - b) : 0ull;
        if (act) {
          any |= fb[s];
          all &= fb[s];
        }
        cand[s] = active[s];
        chosen[s] = 0ull;
      }
      int need = int(R) - wave_reduce_sum_i32(base_sum);
      // +1 for the `need` active positions ranked first by (fraction desc,
      // index asc): a descent over the bits takes positions with the current
      // bit set whole while they fit, else continues among them; bits on
      // which every active position agrees decide nothing
      any = wave_reduce_u64(any, [](uint64_t a, uint64_t b) { return a | b; });
      all = wave_reduce_u64(all, [](uint64_t a, uint64_t b) { return a & b; });
      const int top = (any ^ all) ? 63 - __clzll(any ^ all) : -1;
      for (int bit = top; bit >= 0 && need > 0; --bit) {
        int cnt = 0;
#pragma unroll
        for (int s = 0; s < SL; ++s) cnt += __popcll(cand[s]);
        if (cnt <= need) break;
        uint64_t ones[SL];
        int c1 = 0;
#pragma unroll
        for (int s = 0; s < SL; ++s) {
          ones[s] = cand[s] & __ballot((fb[s] >> bit) & 1ull);
          c1 += __popcll(ones[s]);
        }
        if (c1 <= need) {
#pragma unroll
          for (int s = 0; s < SL; ++s) {
            chosen[s] |= ones[s];
            cand[s] &= ~ones[s];
          }
          need -= c1;
        } else {
#pragma unroll
          for (int s = 0; s < SL; ++s) cand[s] = ones[s];
        }
      }
      // the remaining candidates all fit, or are exact ties: smaller index first
#pragma unroll
      for (int s = 0; s < SL; ++s)
        for (; need > 0 && cand[s]; --need) {
          chosen[s] |= cand[s] & (~cand[s] + 1ull);
          cand[s] &= cand[s] - 1ull;
        }
#pragma unroll
      for (int s = 0; s < SL; ++s)
        if ((chosen[s] >> lane) & 1ull) n[s] += 1;
      R = 0;
    }
  }

  // ---- back to frames, offsets, rectified relevance ----
  int nb[SL];
  double rt[SL];
  if (moved) {
    order();
#pragma unroll
    for (int s = 0; s < SL; ++s) {
      const int i = s * kWave + lane;
      if (i < L) {
        s_nmv[i] = n[s];
        s_mv[0][i] = x[s];
      }
    }
    order();
#pragma unroll
    for (int s = 0; s < SL; ++s) {
      nb[s] = keep[s] ? s_nmv[kpos[s]] : 0;
      rt[s] = keep[s] ? s_mv[0][kpos[s]] : 0.0;
    }
  } else {
#pragma unroll
    for (int s = 0; s < SL; ++s) {
      nb[s] = keep[s] ? n[s] : 0;
      rt[s] = keep[s] ? x[s] : 0.0;
    }
  }
  int carry = 0;
#pragma unroll
  for (int s = 0; s < SL; ++s) {
    const int t = s * kWave + lane;
    const int incl = wave_incl_scan_i32(nb[s]);
    if (t < T) {
      budget[t] = nb[s];
      offset[t] = carry + incl - nb[s];
      if (rel_rect) rel_rect[t] = float(rt[s]);
    }
    carry += __builtin_amdgcn_readlane(incl, kWave - 1);
  }
  if (lane == 0) offset[T] = carry;
}

// Lane t loads r_t and delta_t, then the wave computes the budgets.
__device__ inline void budget_wave_body(const float* __restrict__ rel, const float* __restrict__ delta, int T, int N,
                                        long long B, int levels, float tau, int32_t* __restrict__ budget,
                                        int32_t* __restrict__ offset, float* __restrict__ rel_rect) {
  const int lane = threadIdx.x & 63;
  const double d = lane < T ? double(delta[lane]) : 0.0;
  const double r = lane < T ? double(rel[lane]) : 0.0;
  budget_wave_compute(d, r, T, N, B, levels, tau, budget, offset, rel_rect);
}

}  // namespace
}  // namespace wz
