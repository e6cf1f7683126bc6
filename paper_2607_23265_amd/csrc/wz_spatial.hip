// Stage 3: the per-frame selection that replaces the interpolation of
// Eq. (17), the saliency map M_t (Eq. (7)), the Wavelet Spatial Modulator
// (Eq. (12)-(15)) and the compaction in temporal order (Eq. (19)).  When the
// whole pass runs, stage 2 (the integer budgets, Eq. (9)-(11) and Eq. (16)
// under Eq. (5)) is folded in: every workgroup computes the budgets itself,
// from the same inputs with the same arithmetic, so all of them agree bit for
// bit and no kernel boundary separates the budget from its use.
//
// Workgroup (t, p), p < P, 1024 threads, works on frame t:
//   A. its threads load the frame's scores a_{t,n} as selection keys (larger
//      score first, then the smaller index) and take their min and max;
//      then wave 0 computes the budgets (T <= 64; all waves up to T = 256)
//      while the other waves rank every token of the frame by counting the
//      larger keys (four threads share a token);
//   B. the frame keeps its n_t tokens of rank < n_t; a block-wide count in
//      raster order lists them, with the gate g = lambda * mean(M) of each
//      kept token's 2x2 block, M = min-max of the frame's scores;
//   C. kept tokens p, p + P, ... are reconstructed, each split into channel
//      parts of at most two 16-byte vectors per lane, one part per wave at a
//      time: the 2x2 Haar block of the grid (the last row / column repeated
//      when H or W is odd) is read, LL, LH, HL, HH formed with the
//      orthonormal butterflies (Eq. (12)), the three detail bands multiplied
//      by g (Eq. (13)-(14)) and the token's position inverted (Eq. (15)); the
//      row goes to out_tokens[offset_t + i], its flat index t*H*W + n to
//      out_index.
// Only the blocks of kept tokens are read: at most 4 * B token rows, usually
// partly from the Infinity Cache right after the pass over the frames.
#include "wz_budget.h"

namespace wz {
namespace {

constexpr int kThreads = 1024;
constexpr int kNW = kThreads / kWave;
constexpr int kVecPerLane = 2;  // 16-byte vectors per lane, block row and channel part

enum BudgetSrc : int { kOffsets = 0, kWaveBudget = 1, kBlockBudget = 2 };

struct AssignArgs {
  const void* X;            // [T][H][W][C]
  const float* tok_score;   // [T][H*W] a_{t,n}
  const float* rel;         // [T] r_t        (budget modes)
  const float* delta;       // [T] delta_t    (budget modes)
  const int32_t* offset_in; // [T+1]          (kOffsets)
  int32_t* budget_out;      // [T] or null    (budget modes; written by workgroup (0, 0))
  int32_t* offset_out;      // [T+1] or null  (budget modes)
  void* out_tokens;         // [B][C]
  int32_t* out_index;       // [B]
  long long B;
  int T, H, W, C, P, levels;
  int kpre;  // ranks read before the budget is known (a performance setting)
  float lam, tau;
};

typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// 16 bytes of input: 8 bf16 or 4 fp32 channels, widened to fp32.
template <typename In>
struct Vec16;
template <>
struct Vec16<uint16_t> {
  static constexpr int kV = 8;
  __device__ static void widen(const u32x4& x, float* v) {
#pragma unroll
    for (int i = 0; i < 4; ++i) { v[2 * i] = bf16_lo(x[i]); v[2 * i + 1] = bf16_hi(x[i]); }
  }
};
template <>
struct Vec16<float> {
  static constexpr int kV = 4;
  __device__ static void widen(const u32x4& x, float* v) {
#pragma unroll
    for (int i = 0; i < 4; ++i) v[i] = __uint_as_float(x[i]);
  }
};

template <typename Out, int V>
__device__ __forceinline__ void store_row(Out* p, const float* v);
template <>
__device__ __forceinline__ void store_row<float, 4>(float* p, const float* v) {
  *reinterpret_cast<f32x4*>(p) = f32x4{v[0], v[1], v[2], v[3]};
}
template <>
__device__ __forceinline__ void store_row<float, 8>(float* p, const float* v) {
  reinterpret_cast<f32x4*>(p)[0] = f32x4{v[0], v[1], v[2], v[3]};
  reinterpret_cast<f32x4*>(p)[1] = f32x4{v[4], v[5], v[6], v[7]};
}
template <>
__device__ __forceinline__ void store_row<uint16_t, 8>(uint16_t* p, const float* v) {
  u32x4 o;
#pragma unroll
  for (int i = 0; i < 4; ++i) o[i] = f32_to_bf16_rne(v[2 * i]) | (f32_to_bf16_rne(v[2 * i + 1]) << 16);
  *reinterpret_cast<u32x4*>(p) = o;
}
template <>
__device__ __forceinline__ void store_row<uint16_t, 4>(uint16_t* p, const float* v) {
  u32x2 o;
  o[0] = f32_to_bf16_rne(v[0]) | (f32_to_bf16_rne(v[1]) << 16);
  o[1] = f32_to_bf16_rne(v[2]) | (f32_to_bf16_rne(v[3]) << 16);
  *reinterpret_cast<u32x2*>(p) = o;
}

constexpr int kBins = 256;  // score bins of the ranking

template <typename In, typename Out, int U, int MODE>
__global__ __launch_bounds__(kThreads) void k_assign_gather(const AssignArgs f) {
  constexpr int V = Vec16<In>::kV;
  // The ranking group: every wave but wave 0 when wave 0 computes the
  // budgets meanwhile (kWaveBudget), else all waves.
  constexpr int G0 = MODE == kWaveBudget ? 1 : 0;
  constexpr int GW = kNW - G0;
  extern __shared__ __align__(16) char s_dyn[];
  __shared__ int32_t s_nb[kFusedTMax];       // budgets (budget modes)
  __shared__ int32_t s_off[kFusedTMax + 1];  // offsets (budget modes)
  __shared__ float s_mm[2][kNW];             // per-wave min / max of the scores
  __shared__ int s_cnt[kNW];
  __shared__ int s_start[kBins];             // first sorted position of each bin (bins in descending order)
  __shared__ int s_fill[kBins];              // tokens per bin
  __shared__ int s_sync;                     // arrivals at the ranking group's barriers

  const int N = f.H * f.W, T = f.T;
  const int b = blockIdx.x, xcd = b % kXcds, slot = b / kXcds;
  const int t = (slot / f.P) * kXcds + xcd, p = slot % f.P;
  if (t >= T) return;  // whole workgroup
  uint64_t* s_key = reinterpret_cast<uint64_t*>(s_dyn);     // [N] selection keys
  int32_t* s_rank = reinterpret_cast<int32_t*>(s_key + N);  // [N] rank of each token
  int32_t* s_byrank = s_rank + N;                           // [N] token of each rank
  int32_t* s_posr = s_byrank + N;                           // [N] raster position among the kept, by rank
  float* s_gate = reinterpret_cast<float*>(s_posr + N);     // [N] gate of each token's block
  int32_t* s_sorted = s_posr;                               // [N] tokens by bin (before the positions)
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int gi = tid - G0 * kWave, gn = GW * kWave;         // thread index and count in the group

  // budget inputs first: wave 0 computes the budgets as soon as they arrive
  double bd = 0.0, br = 0.0;
  int o_base = 0, o_next = 0, o_last = 0;
  if constexpr (MODE == kWaveBudget) {
    if (wave == 0 && lane < T) {
      bd = double(f.delta[lane]);
      br = double(f.rel[lane]);
    }
  } else if constexpr (MODE == kOffsets) {
    o_base = f.offset_in[t];
    o_next = f.offset_in[t + 1];
    o_last = f.offset_in[T];
  }
  if (tid == 0) s_sync = 0;
  lds_barrier();

  // Barrier of the ranking group alone (wave 0 may be inside the budget): an
  // arrival counter in LDS that every group wave increments once per barrier
  // and waits on; every group wave reaches every such barrier.
  int gen = 0;
  auto group_sync = [&]() {
    if constexpr (MODE == kWaveBudget) {
      ++gen;
      if (lane == 0) __hip_atomic_fetch_add(&s_sync, 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
      while (__hip_atomic_load(&s_sync, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP) < gen * GW)
        __builtin_amdgcn_s_sleep(1);
    } else {
      lds_barrier();
    }
  };

  // Channel parts of a kept token: at most U vectors per lane each.
  const int nvec = f.C / V;
  const int parts = (nvec + U * kWave - 1) / (U * kWave);
  const int vpp = (nvec + parts - 1) / parts;  // vectors per part
  const int rb = f.C * int(sizeof(In));
  const __amdgpu_buffer_rsrc_t xres = make_rsrc(static_cast<const In*>(f.X) + size_t(t) * N * f.C, uint32_t(N) * rb);
  // This workgroup reconstructs the kept tokens of rank p, p + P, ...; item j
  // is part j % parts of the token of rank p + P * (j / parts).  The first
  // items, up to one per group wave and for ranks below kpre (where most
  // frames' budgets reach), are read before the budget is known.
  const int kp = min(f.kpre, N);
  const int npre = MODE == kWaveBudget && kp > p ? min(GW, (kp - p + f.P - 1) / f.P * parts) : 0;
  u32x4 xp[U][4];
  auto load_item = [&](int j, u32x4 (&x)[U][4]) {
    const int n = s_byrank[p + f.P * (j / parts)];
    const int h = n / f.W, w = n - h * f.W;
    const int i0 = h & ~1, j0 = w & ~1;
    const int i1 = min(i0 + 1, f.H - 1), j1 = min(j0 + 1, f.W - 1);
    const int r00 = (i0 * f.W + j0) * rb, r01 = (i0 * f.W + j1) * rb;
    const int r10 = (i1 * f.W + j0) * rb, r11 = (i1 * f.W + j1) * rb;
    const int vb = (j % parts) * vpp, ve = min(nvec, vb + vpp);
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int v = vb + u * kWave + lane;
      const int cb = v < ve ? v * 16 : kOOB;
      x[u][0] = __builtin_amdgcn_raw_buffer_load_b128(xres, r00 + cb, 0, 0);
      x[u][1] = __builtin_amdgcn_raw_buffer_load_b128(xres, r01 + cb, 0, 0);
      x[u][2] = __builtin_amdgcn_raw_buffer_load_b128(xres, r10 + cb, 0, 0);
      x[u][3] = __builtin_amdgcn_raw_buffer_load_b128(xres, r11 + cb, 0, 0);
    }
  };

  if constexpr (MODE == kWaveBudget) {
    if (wave == 0) budget_wave_compute(bd, br, T, N, f.B, f.levels, f.tau, s_nb, s_off, nullptr);
  } else if constexpr (MODE == kBlockBudget) {
    budget_body<kThreads, kFusedTMax>(f.rel, f.delta, T, N, f.B, f.levels, f.tau, s_nb, s_off, nullptr);
  }

  if (wave >= G0) {
    // ---- A. the frame's scores as selection keys (larger score first, then
    // the smaller index), their extremes, and the ranks by bins of score ----
    const __amdgpu_buffer_rsrc_t ares = make_rsrc(f.tok_score + size_t(t) * N, uint32_t(N) * 4);
    float lo = INFINITY, hi = -INFINITY;
    for (int n0 = 0; n0 < N; n0 += 4 * gn) {
      float av[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int n = n0 + u * gn + gi;
        av[u] = buf_load_f32(ares, n < N ? n * 4 : kOOB);
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int n = n0 + u * gn + gi;
        if (n < N) {
          s_key[n] = sel_key(av[u], n);
          lo = fminf(lo, av[u]);
          hi = fmaxf(hi, av[u]);
        }
      }
    }
    for (int q = gi; q < kBins; q += gn) s_fill[q] = 0;
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) {
      lo = fminf(lo, __shfl_xor(lo, m, kWave));
      hi = fmaxf(hi, __shfl_xor(hi, m, kWave));
    }
    if (lane == 0) {
      s_mm[0][wave] = lo;
      s_mm[1][wave] = hi;
    }
    group_sync();
    lo = s_mm[0][G0];
    hi = s_mm[1][G0];
#pragma unroll
    for (int w = G0 + 1; w < kNW; ++w) {
      lo = fminf(lo, s_mm[0][w]);
      hi = fmaxf(hi, s_mm[1][w]);
    }
    const float range = hi - lo;
    // bin of a score: linear in the score between the extremes, so never
    // lower for a larger selection key (NaN keys sort outside every number
    // and go to the end bins; without a finite positive range every number
    // shares bin 0)
    const float bscale = range > 0.f && range < INFINITY ? float(kBins) / range : 0.f;
    auto bin_of = [&](uint64_t key) {
      const float a = order_value(uint32_t(key >> 12));
      if (a != a) return (key >> 43) ? kBins - 1 : 0;
      return min(kBins - 1, max(0, int((a - lo) * bscale)));
    };
    for (int n = gi; n < N; n += gn) atomicAdd(&s_fill[bin_of(s_key[n])], 1);
    group_sync();
    if (wave == G0) {
      // start of bin q = tokens in bins above q: a scan over the bins from the top
      int c[kBins / kWave], sum = 0;
#pragma unroll
      for (int e = 0; e < kBins / kWave; ++e) {
        c[e] = s_fill[kBins - 1 - (lane * (kBins / kWave) + e)];
        sum += c[e];
      }
      int incl = sum;
#pragma unroll
      for (int d = 1; d < kWave; d <<= 1) {
        const int o = __shfl_up(incl, d, kWave);
        if (lane >= d) incl += o;
      }
      int run = incl - sum;
#pragma unroll
      for (int e = 0; e < kBins / kWave; ++e) {
        const int q = kBins - 1 - (lane * (kBins / kWave) + e);
        s_start[q] = run;
        run += c[e];
        s_fill[q] = 0;
      }
    }
    group_sync();
    for (int n = gi; n < N; n += gn) {
      const int q = bin_of(s_key[n]);
      s_sorted[s_start[q] + atomicAdd(&s_fill[q], 1)] = n;
    }
    group_sync();
    // rank = tokens in higher bins + larger keys in the same bin
    for (int n = gi; n < N; n += gn) {
      const uint64_t kn = s_key[n];
      const int q = bin_of(kn);
      const int j0 = s_start[q], j1 = j0 + s_fill[q];
      int r = j0;
      for (int j = j0; j < j1; ++j) r += s_key[s_sorted[j]] > kn;
      s_rank[n] = r;
      s_byrank[r] = n;
    }
    // gate g = lambda * mean(M) of the 2x2 block of each token (Eq. (13)),
    // M = min-max of the frame's scores (Eq. (7))
    auto sal = [&](int n) {
      const float a = order_value(uint32_t(s_key[n] >> 12));
      return range > 0.f ? (a - lo) / range : 0.f;
    };
    for (int n = gi; n < N; n += gn) {
      const int h = n / f.W, w = n - h * f.W;
      const int i0 = h & ~1, j0 = w & ~1;
      const int i1 = min(i0 + 1, f.H - 1), j1 = min(j0 + 1, f.W - 1);
      const float m00 = sal(i0 * f.W + j0), m01 = sal(i0 * f.W + j1), m10 = sal(i1 * f.W + j0),
                  m11 = sal(i1 * f.W + j1);
      s_gate[n] = f.lam * (0.25f * (((m00 + m01) + m10) + m11));
    }
    group_sync();  // every rank known: the first items' reads go out
    if (wave - G0 < npre) load_item(wave - G0, xp);
  }
  // LDS-only barriers from here on: the prefetch reads stay in flight
  lds_barrier();  // ranks, gates and budgets published

  long long base, total;
  int nt;
  if constexpr (MODE == kOffsets) {
    base = o_base;
    nt = min(o_next - o_base, N);
    total = min((long long)o_last, f.B);
  } else {
    base = s_off[t];
    nt = s_off[t + 1] - s_off[t];
    total = s_off[T];
    if (t == 0 && p == 0) {
      for (int i = tid; i < T; i += kThreads) {
        if (f.budget_out) f.budget_out[i] = s_nb[i];
        if (f.offset_out) f.offset_out[i] = s_off[i];
      }
      if (tid == 0 && f.offset_out) f.offset_out[T] = s_off[T];
    }
  }

  // ---- B. raster positions of the kept tokens (ballots, one token per thread and round) ----
  int run = 0;  // kept tokens of earlier rounds
  for (int n0 = 0; n0 < N; n0 += kThreads) {
    const int n = n0 + tid;
    const int r = n < N ? s_rank[n] : 0;
    const bool kept = n < N && r < nt;
    const uint64_t m = __ballot(kept);
    if (lane == 0) s_cnt[wave] = __popcll(m);
    lds_barrier();
    int before = run, tot = 0;
#pragma unroll
    for (int w = 0; w < kNW; ++w) {
      const int cw = s_cnt[w];
      before += w < wave ? cw : 0;
      tot += cw;
    }
    if (kept) s_posr[r] = before + __popcll(m & ((1ull << lane) - 1ull));
    run += tot;
    lds_barrier();
  }

  // ---- C. reconstruction of the kept tokens of rank p, p + P, ... ----
  const int mine = nt > p ? (nt - p + f.P - 1) / f.P : 0;  // kept tokens of this workgroup
  auto finish_item = [&](int j, const u32x4 (&x)[U][4]) {
    const int r = p + f.P * (j / parts);
    const long long k = base + s_posr[r];
    if (k < 0 || k >= total) return;
    const int n = s_byrank[r];
    const float g = s_gate[n];
    const int h = n / f.W, w = n - h * f.W;
    const float sw = (w & 1) ? -1.f : 1.f;
    const float sh = (h & 1) ? -1.f : 1.f;
    Out* dst = static_cast<Out*>(f.out_tokens) + size_t(k) * f.C;
    const int vb = (j % parts) * vpp, ve = min(nvec, vb + vpp);
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int v = vb + u * kWave + lane;
      float x00[V], x01[V], x10[V], x11[V], y[V];
      Vec16<In>::widen(x[u][0], x00);
      Vec16<In>::widen(x[u][1], x01);
      Vec16<In>::widen(x[u][2], x10);
      Vec16<In>::widen(x[u][3], x11);
#pragma unroll
      for (int e = 0; e < V; ++e) {
        // orthonormal 2-D Haar butterflies of the block (Eq. (12))
        const float LL = 0.5f * ((x00[e] + x01[e]) + (x10[e] + x11[e]));
        const float LH = 0.5f * ((x00[e] - x01[e]) + (x10[e] - x11[e]));
        const float HL = 0.5f * ((x00[e] + x01[e]) - (x10[e] + x11[e]));
        const float HH = 0.5f * ((x00[e] - x01[e]) - (x10[e] - x11[e]));
        // gate the detail bands (Eq. (14)) and invert at the token's position (Eq. (15))
        y[e] = 0.5f * (LL + g * (sw * LH + sh * HL + (sw * sh) * HH));
      }
      if (v < ve) store_row<Out, V>(dst + v * V, y);
    }
    if (j % parts == 0 && lane == 0) f.out_index[k] = t * N + n;
  };
  // prefetched items whose token is kept, then the rest
  if (wave >= G0 && wave - G0 < npre && wave - G0 < mine * parts) finish_item(wave - G0, xp);
  for (int j = npre + wave; j < mine * parts; j += kNW) {
    u32x4 x[U][4];
    load_item(j, x);
    finish_item(j, x);
  }
}

template <typename In, typename Out, int MODE>
void launch_typed(const wz_config& c, const AssignArgs& a, hipStream_t s) {
  const int nvec = c.C / Vec16<In>::kV;
  const dim3 grid(unsigned((c.T + kXcds - 1) / kXcds * kXcds * a.P)), block(kThreads);
  const size_t lds = size_t(c.H) * c.W * 24;  // keys (8 B); rank, token by rank, position, gate (4 B each)
  // one batch of loads per part: two vectors per lane, or one for short rows
  if (nvec <= kWave) hipLaunchKernelGGL((k_assign_gather<In, Out, 1, MODE>), grid, block, lds, s, a);
  else hipLaunchKernelGGL((k_assign_gather<In, Out, kVecPerLane, MODE>), grid, block, lds, s, a);
}

template <int MODE>
void launch_mode(const wz_config& c, const AssignArgs& a, hipStream_t s) {
  if (c.in_dtype == WZ_BF16) {
    if (c.out_dtype == WZ_BF16) launch_typed<uint16_t, uint16_t, MODE>(c, a, s);
    else launch_typed<uint16_t, float, MODE>(c, a, s);
  } else {
    if (c.out_dtype == WZ_BF16) launch_typed<float, uint16_t, MODE>(c, a, s);
    else launch_typed<float, float, MODE>(c, a, s);
  }
}

}  // namespace

int assign_groups_per_frame(const wz_config& c) {
  // about one workgroup per CU over the whole grid, at most 16 per frame;
  // each repeats its frame's ranking (N^2 key comparisons), so large frames
  // get fewer
  const int tr = (c.T + kXcds - 1) / kXcds * kXcds;
  const int cap = std::max(1, std::min(16, 8192 / (c.H * c.W)));
  return std::max(1, std::min(cap, (kCUs + tr - 1) / tr));
}

hipError_t launch_assign_gather(const wz_config& c, const void* X, const float* tok_score, const float* frame_rel,
                                const float* frame_delta, const int32_t* offset_in, int32_t* budget_out,
                                int32_t* offset_out, void* out_tokens, int32_t* out_index, hipStream_t s) {
  // three quarters of the mean budget: most frames keep at least that many
  const int kpre = int(std::min<long long>(c.H * c.W, 3 * c.B / (4LL * c.T)));
  AssignArgs a{X,         tok_score, frame_rel, frame_delta, offset_in, budget_out, offset_out, out_tokens,
               out_index, c.B,       c.T,       c.H,         c.W,       c.C,        assign_groups_per_frame(c),
               c.levels,  kpre,      c.lambda_, c.tau};
  if (offset_in) launch_mode<kOffsets>(c, a, s);
  else if (c.T <= kWave) launch_mode<kWaveBudget>(c, a, s);
  else if (c.T <= kFusedTMax) launch_mode<kBlockBudget>(c, a, s);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace wz
