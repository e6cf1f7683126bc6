// Selection order of one frame's tokens and the saliency gates of their 2x2
// blocks, computed by one workgroup with the frame in LDS:
//   key_n  = (score order, complemented index): larger score first, then the
//            smaller index, so keys are distinct (the selection that replaces
//            Eq. (17) keeps the n_t largest keys);
//   rank_n = number of keys larger than key_n (byrank inverts it);
//   gate_n = lambda * mean of M over the 2x2 block of token n (Eq. (13)),
//            M = min-max of the frame's scores (Eq. (7)), 0 when all equal;
//            the last row / column is repeated when H or W is odd;
//   gate2_n (two spatial levels) = lambda * mean of those block means over
//            the 2x2 blocks of blocks around token n, repeated at the edge
//            likewise.
// Ranks come from a counting sort into score bins (linear in the score
// between the frame's extremes, so a larger key never lands in a lower bin)
// and a comparison of the keys that share a bin.
#pragma once

#include "wz_device.h"

namespace wz {
namespace {

constexpr int kBins = 256;

struct RankLds {  // LDS arrays of the frame
  uint64_t* key;    // [N], filled by the caller
  int32_t* rank;    // [N]
  int32_t* byrank;  // [N]
  float* gate;      // [N]
  float* gate2;     // [N] level-2 gates (two spatial levels), or null
  int32_t* order;   // [N] scratch: tokens in bin order
  int* start;       // [kBins] first position of each bin, bins from the top
  int* fill;        // [kBins]
  float* mm;        // [2 * NTH / 64] per-wave extremes
};

// All NTH threads of the workgroup call this once the keys are written to
// s.key (no barrier needed before the call); lo / hi are each thread's
// extremes over the scores it wrote.  Ends without a trailing barrier.
template <int NTH>
__device__ void rank_frame(int N, int H, int W, float lam, float lo, float hi, const RankLds& s) {
  constexpr int NW = NTH / kWave;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  lo = wave_min_f32(lo);
  hi = wave_max_f32(hi);
  if (lane == 0) {
    s.mm[wave] = lo;
    s.mm[NW + wave] = hi;
  }
  for (int q = tid; q < kBins; q += NTH) s.fill[q] = 0;
  lds_barrier();
  lo = s.mm[0];
  hi = s.mm[NW];
#pragma unroll
  for (int w = 1; w < NW; ++w) {
    lo = fminf(lo, s.mm[w]);
    hi = fmaxf(hi, s.mm[NW + w]);
  }
  const float range = hi - lo;
  // NaN keys sort outside every number and go to the end bins; without a
  // finite positive range every number shares bin 0
  const float bscale = range > 0.f && range < INFINITY ? float(kBins) / range : 0.f;
  auto bin_of = [&](uint64_t key) {
    const float a = order_value(uint32_t(key >> 12));
    if (a != a) return (key >> 43) ? kBins - 1 : 0;
    return min(kBins - 1, max(0, int((a - lo) * bscale)));
  };
  for (int n = tid; n < N; n += NTH) atomicAdd(&s.fill[bin_of(s.key[n])], 1);
  lds_barrier();
  if (wave == 0) {
    // start of bin q = tokens in the bins above it
    constexpr int PL = kBins / kWave;
    int c[PL], sum = 0;
#pragma unroll
    for (int e = 0; e < PL; ++e) {
      c[e] = s.fill[kBins - 1 - (lane * PL + e)];
      sum += c[e];
    }
    int run = wave_incl_scan_i32(sum) - sum;
#pragma unroll
    for (int e = 0; e < PL; ++e) {
      const int q = kBins - 1 - (lane * PL + e);
      s.start[q] = run;
      run += c[e];
      s.fill[q] = 0;
    }
  }
  lds_barrier();
  for (int n = tid; n < N; n += NTH) {
    const int q = bin_of(s.key[n]);
    s.order[s.start[q] + atomicAdd(&s.fill[q], 1)] = n;
  }
  lds_barrier();
  for (int n = tid; n < N; n += NTH) {
    const uint64_t kn = s.key[n];
    const int q = bin_of(kn);
    const int j0 = s.start[q], j1 = j0 + s.fill[q];
    int r = j0;
    for (int j = j0; j < j1; ++j) r += s.key[s.order[j]] > kn;
    s.rank[n] = r;
    s.byrank[r] = n;
  }
  auto sal = [&](int n) {
    const float a = order_value(uint32_t(s.key[n] >> 12));
    return range > 0.f ? (a - lo) / range : 0.f;
  };
  for (int n = tid; n < N; n += NTH) {
    const int h = n / W, w = n - h * W;
    const int i0 = h & ~1, j0 = w & ~1;
    const int i1 = min(i0 + 1, H - 1), j1 = min(j0 + 1, W - 1);
    const float m00 = sal(i0 * W + j0), m01 = sal(i0 * W + j1), m10 = sal(i1 * W + j0), m11 = sal(i1 * W + j1);
    s.gate[n] = lam * (0.25f * (((m00 + m01) + m10) + m11));
  }
  if (s.gate2) {
    // two spatial levels: lambda * the mean of M over the level-1 cells (2x2
    // token blocks) of the token's level-2 block, the last cell / token row
    // and column repeated at each level
    const int Hb = (H + 1) / 2, Wb = (W + 1) / 2;
    auto cell = [&](int bi, int bj) {
      const int i0 = 2 * bi, j0 = 2 * bj, i1 = min(i0 + 1, H - 1), j1 = min(j0 + 1, W - 1);
      return 0.25f * (((sal(i0 * W + j0) + sal(i0 * W + j1)) + sal(i1 * W + j0)) + sal(i1 * W + j1));
    };
    for (int n = tid; n < N; n += NTH) {
      const int h = n / W, w = n - h * W;
      const int c0 = 2 * (h / 4), d0 = 2 * (w / 4), c1 = min(c0 + 1, Hb - 1), d1 = min(d0 + 1, Wb - 1);
      s.gate2[n] = lam * (0.25f * (((cell(c0, d0) + cell(c0, d1)) + cell(c1, d0)) + cell(c1, d1)));
    }
  }
}

}  // namespace
}  // namespace wz
