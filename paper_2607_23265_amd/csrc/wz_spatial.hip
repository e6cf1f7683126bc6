// Stage 3: the per-frame selection that replaces the interpolation of
// Eq. (17), the saliency map M_t (Eq. (7)), the Wavelet Spatial Modulator
// (Eq. (12)-(15)) and the compaction in temporal order (Eq. (19)).  When the
// whole pass runs, stage 2 (the integer budgets, Eq. (9)-(11) and Eq. (16)
// under Eq. (5)) is folded in: every workgroup computes the budgets itself,
// from the same inputs with the same arithmetic, so all of them agree bit for
// bit and no kernel boundary separates the budget from its use.
//
// Workgroup (t, p), p < P, 1024 threads, works on frame t:
//   A. wave 0 computes the budgets (T <= 256: in registers, one frame per
//      lane up to 64 frames, four above; beyond 256 they come from the
//      budget kernel launched before this one) while
//      the other waves take the frame's selection ranks and block gates
//      (from the per-frame kernel, or formed here from the scores when the
//      stage runs on its own, wz_rank.h) and form the rows of the first
//      tokens this workgroup will emit: most frames keep at least three
//      quarters of the mean budget, so that work is rarely wasted and it
//      overlaps the budget;
//   B. the frame keeps its n_t tokens of rank < n_t.  Each token is emitted
//      in channel parts of at most two 16-byte vectors per lane, one part per
//      wave at a time.  The read-ahead rows go out first; the kept tokens of
//      higher rank of ALL frames are then shared out evenly over all
//      workgroups (every workgroup knows every budget), so frames with large
//      budgets do not leave a few CUs working alone.  With the offsets given
//      (T > 256, or the stage on its own) each workgroup emits its frame's
//      kept tokens of rank p, p + P, ... instead, the next part's block reads
//      in flight while one is finished.  A token's row is its 2x2 Haar block
//      (the last row / column repeated when H or W is odd) through the
//      orthonormal butterflies (Eq. (12)), the three detail bands multiplied
//      by the block's gate (Eq. (13)-(14)) and the inverse at the token's
//      position (Eq. (15)), evaluated in the equivalent form mu + g (x - mu),
//      mu the block mean.  It goes to out_tokens[offset_t + position],
//      position = kept tokens before it in raster order (a wave's own
//      ballots over the ranks), its flat index t*H*W + n to out_index.
// Two further ways to form the rows (kernel parameter AM): the budget-guided
// interpolation of Eq. (17) (cfg.assign = WZ_INTERP: each of a frame's n_t
// cells blends four modulated taps of the frame), and the two-level spatial
// modulator (cfg.spatial_levels = 2: a kept token's row from its 4x4 level-2
// block).  Their cells depend on the budget or read 16 rows, so they read
// nothing ahead and share every output row out over all workgroups.
// Only the blocks of kept tokens are read: at most 4 * B token rows (16 * B
// for the interpolation and two levels), partly from the Infinity Cache right
// after the pass over the frames.
#include "wz_budget.h"
#include "wz_rank.h"

namespace wz {
namespace {

constexpr int kThreads = 1024;
constexpr int kNW = kThreads / kWave;
constexpr int kVecPerLane = 2;  // 16-byte vectors per lane, block row and channel part

enum BudgetSrc : int { kOffsets = 0, kWaveBudget = 1 };

struct AssignArgs {
  const void* X;            // [T][H][W][C]
  const float* tok_score;   // [T][H*W] a_{t,n}
  const float* rel;         // [T] r_t        (budget modes)
  const float* delta;       // [T] delta_t    (budget modes)
  const int32_t* offset_in; // [T+1]          (kOffsets)
  const int32_t* rank;      // [T][H*W] or null: selection ranks from the per-frame kernel
  const int32_t* byrank;    // [T][H*W]
  const float* gate;        // [T][H*W]
  const float* gate2;       // [T][H*W] level-2 gates (two spatial levels, with the per-frame kernel)
  int32_t* budget_out;      // [T] or null    (budget modes; written by workgroup (0, 0))
  int32_t* offset_out;      // [T+1] or null  (budget modes)
  void* out_tokens;         // [B][C]
  int32_t* out_index;       // [B]
  long long B;
  int T, H, W, C, P, levels;
  int kpre;  // ranks read before the budget is known (a performance setting)
  float lam, tau;
};
static_assert(sizeof(VideoArgs<AssignArgs>) <= 4096, "per-video arguments exceed the kernel argument limit");

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

// One row vector of the output (16 bytes of input widened to V floats), at
// byte offset off of the row's buffer, written through the L2.
template <typename Out, int V>
__device__ __forceinline__ void store_row(__amdgpu_buffer_rsrc_t r, int off, const float* v);
template <>
__device__ __forceinline__ void store_row<float, 4>(__amdgpu_buffer_rsrc_t r, int off, const float* v) {
  buf_store_wt_b128(u32x4{__float_as_uint(v[0]), __float_as_uint(v[1]), __float_as_uint(v[2]), __float_as_uint(v[3])},
                    r, off);
}
template <>
__device__ __forceinline__ void store_row<float, 8>(__amdgpu_buffer_rsrc_t r, int off, const float* v) {
  buf_store_wt_b128(u32x4{__float_as_uint(v[0]), __float_as_uint(v[1]), __float_as_uint(v[2]), __float_as_uint(v[3])},
                    r, off);
  buf_store_wt_b128(u32x4{__float_as_uint(v[4]), __float_as_uint(v[5]), __float_as_uint(v[6]), __float_as_uint(v[7])},
                    r, off + 16);
}
template <>
__device__ __forceinline__ void store_row<uint16_t, 8>(__amdgpu_buffer_rsrc_t r, int off, const float* v) {
  u32x4 o;
#pragma unroll
  for (int i = 0; i < 4; ++i) o[i] = f32_to_bf16_rne(v[2 * i]) | (f32_to_bf16_rne(v[2 * i + 1]) << 16);
  buf_store_wt_b128(o, r, off);
}
template <>
__device__ __forceinline__ void store_row<uint16_t, 4>(__amdgpu_buffer_rsrc_t r, int off, const float* v) {
  const uint64_t lo = f32_to_bf16_rne(v[0]) | (f32_to_bf16_rne(v[1]) << 16);
  const uint64_t hi = f32_to_bf16_rne(v[2]) | (f32_to_bf16_rne(v[3]) << 16);
  buf_store_wt_b64(lo | (hi << 32), r, off);
}

// AM: how the rows are formed -- kSelect1 (selection, one spatial level),
// kInterp (budget-guided interpolation), kSelect2 (selection, two levels).
enum AssignMode : int { kSelect1 = 0, kInterp = 1, kSelect2 = 2 };

template <typename In, typename Out, int U, int MODE, int AM>
__global__ __launch_bounds__(kThreads) void k_assign_gather(const VideoArgs<AssignArgs> va) {
  constexpr bool INTERP = AM == kInterp, L2 = AM == kSelect2;
  const AssignArgs& f = va.v[blockIdx.y];
  constexpr int V = Vec16<In>::kV;
  // waves that read ranks and blocks while wave 0 computes the budgets
  constexpr int G0 = MODE == kWaveBudget ? 1 : 0;
  constexpr int GW = kNW - G0;
  extern __shared__ __align__(16) char s_dyn[];
  __shared__ int32_t s_nb[kFusedTMax];       // budgets (budget modes)
  __shared__ int32_t s_off[kFusedTMax + 1];  // offsets (budget modes)
  __shared__ int32_t s_ext[kFusedTMax + 1];  // kept tokens of rank >= kp in the frames before t (budget modes)
  __shared__ float s_mm[2 * kNW];
  __shared__ int s_start[kBins], s_fill[kBins];

  const int N = f.H * f.W, T = f.T;
  const int b = blockIdx.x, xcd = b % kXcds, slot = b / kXcds;
  const int t = (slot / f.P) * kXcds + xcd, p = slot % f.P;
  if (t >= T) return;  // whole workgroup
  RankLds rl;
  rl.key = reinterpret_cast<uint64_t*>(s_dyn);
  rl.rank = reinterpret_cast<int32_t*>(rl.key + N);
  rl.byrank = rl.rank + N;
  rl.gate = reinterpret_cast<float*>(rl.byrank + N);
  rl.order = reinterpret_cast<int32_t*>(rl.gate + N);
  rl.gate2 = L2 ? reinterpret_cast<float*>(rl.order + N) : nullptr;
  rl.start = s_start;
  rl.fill = s_fill;
  rl.mm = s_mm;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const bool given = f.rank != nullptr;

  // Channel parts of a kept token: at most U vectors per lane each.
  const int nvec = f.C / V;
  const int parts = (nvec + U * kWave - 1) / (U * kWave);
  const int vpp = (nvec + parts - 1) / parts;  // vectors per part
  const int rb = f.C * int(sizeof(In));
  const __amdgpu_buffer_rsrc_t xres = make_rsrc(static_cast<const In*>(f.X) + size_t(t) * N * f.C, uint32_t(N) * rb);
  // This workgroup reconstructs the kept tokens of rank p, p + P, ...; item j
  // is part j % parts of the token of rank p + P * (j / parts).  The first
  // items, one per reading wave and for ranks below kpre, are read before the
  // budget is known.
  // ranks below kp are read ahead (before the budget), each by its frame's
  // workgroup p = rank mod P, one item per reading wave
  const int kp = given && AM == kSelect1 ? min(min(f.kpre, N), f.P * (GW / parts)) : 0;
  const int npre = kp > p ? (kp - p + f.P - 1) / f.P * parts : 0;
  // the four rows of token n's 2x2 block, the token's own row first: the
  // block's other row h2 and column w2 (the last row / column repeated when
  // H or W is odd)
  auto load_rows = [&](__amdgpu_buffer_rsrc_t xr, int part, int n, u32x4 (&x)[U][4]) {
    const int h = n / f.W, w = n - h * f.W;
    const int h2 = (h & 1) ? h - 1 : min(h + 1, f.H - 1), w2 = (w & 1) ? w - 1 : min(w + 1, f.W - 1);
    const int r0 = (h * f.W + w) * rb, r1 = (h * f.W + w2) * rb;
    const int r2 = (h2 * f.W + w) * rb, r3 = (h2 * f.W + w2) * rb;
    const int vb = part * vpp, ve = min(nvec, vb + vpp);
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int v = vb + u * kWave + lane;
      const int cb = v < ve ? v * 16 : kOOB;
      x[u][0] = __builtin_amdgcn_raw_buffer_load_b128(xr, r0 + cb, 0, 0);
      x[u][1] = __builtin_amdgcn_raw_buffer_load_b128(xr, r1 + cb, 0, 0);
      x[u][2] = __builtin_amdgcn_raw_buffer_load_b128(xr, r2 + cb, 0, 0);
      x[u][3] = __builtin_amdgcn_raw_buffer_load_b128(xr, r3 + cb, 0, 0);
    }
  };
  auto load_item = [&](int j, int n, u32x4 (&x)[U][4]) { load_rows(xres, j % parts, n, x); };

  // ---- A. budgets; ranks and gates; the first blocks ----
  double bd = 0.0, br = 0.0;
  int o_base = 0, o_next = 0, o_last = 0;
  if constexpr (MODE == kWaveBudget) {
    if (wave == 0 && lane < T) {
      bd = double(f.delta[lane]);
      br = double(f.rel[lane]);
    }
  } else {
    o_base = f.offset_in[t];
    o_next = f.offset_in[t + 1];
    o_last = f.offset_in[T];
  }
  // The gated 2x2 Haar round trip of a token, for the channel part in x:
  // the orthonormal butterflies of its block (Eq. (12)), the three detail
  // bands times the gate g (Eq. (13)-(14)) and the inverse at the token's own
  // position (Eq. (15)) come to mu + g (x - mu), mu the block mean: the
  // approximation band alone synthesises mu at every position and the detail
  // bands alone x - mu.  x[.][0] is the token's own row.
  auto modulate = [&](const u32x4 (&x)[U][4], float g, float (&y)[U][V]) {
    const float c = 0.25f * (1.f - g);
#pragma unroll
    for (int u = 0; u < U; ++u) {
      float x0[V], x1[V], x2[V], x3[V];
      Vec16<In>::widen(x[u][0], x0);
      Vec16<In>::widen(x[u][1], x1);
      Vec16<In>::widen(x[u][2], x2);
      Vec16<In>::widen(x[u][3], x3);
#pragma unroll
      for (int e = 0; e < V; ++e) y[u][e] = fmaf(c, (x0[e] + x1[e]) + (x2[e] + x3[e]), g * x0[e]);
    }
  };
  // kept tokens (rank < nt) before token n in raster order: ballots over the
  // frame's ranks in LDS, by the calling wave alone
  auto position = [&](int n, int nt) {
    int before = 0;
    for (int m0 = 0; m0 < n; m0 += kWave) {
      const int m = m0 + lane;
      before += __popcll(__ballot(m < n && rl.rank[m] < nt));
    }
    return before;
  };
  // Two spatial levels: the 16 rows of the four level-1 cells (2x2 token
  // blocks) of token n's level-2 block, the token's own cell first with its
  // own row first (the last row / column repeated at each level), then
  //   x~ = mu2 + g2 (mu1 - mu2) + g1 (x - mu1),
  // mu1 the mean of the token's cell, mu2 the mean of the four cell means:
  // what the two-level butterflies with gated details come to.
  auto load_rows2 = [&](__amdgpu_buffer_rsrc_t xr, int part, int n, u32x4 (&x)[4][U][4]) {
    const int Hb = (f.H + 1) / 2, Wb = (f.W + 1) / 2;
    const int h = n / f.W, w = n - h * f.W, bi = h / 2, bj = w / 2;
    const int bi2 = (bi & 1) ? bi - 1 : min(bi + 1, Hb - 1), bj2 = (bj & 1) ? bj - 1 : min(bj + 1, Wb - 1);
    load_rows(xr, part, n, x[0]);
    const int cells[3][2] = {{bi, bj2}, {bi2, bj}, {bi2, bj2}};
#pragma unroll
    for (int q = 0; q < 3; ++q) {
      const int ci = cells[q][0], cj = cells[q][1];
      load_rows(xr, part, (2 * ci) * f.W + 2 * cj, x[q + 1]);  // the cell's four tokens
    }
  };
  auto modulate2 = [&](const u32x4 (&x)[4][U][4], float g1, float g2, float (&y)[U][V]) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      float r[4][4][V];
#pragma unroll
      for (int q = 0; q < 4; ++q)
#pragma unroll
        for (int k = 0; k < 4; ++k) Vec16<In>::widen(x[q][u][k], r[q][k]);
#pragma unroll
      for (int e = 0; e < V; ++e) {
        float m[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) m[q] = 0.25f * (((r[q][0][e] + r[q][1][e]) + r[q][2][e]) + r[q][3][e]);
        const float mu2 = 0.25f * (((m[0] + m[1]) + m[2]) + m[3]);
        y[u][e] = mu2 + g2 * (m[0] - mu2) + g1 * (r[0][0][e] - m[0]);
      }
    }
  };

  // row k of the output: channel part `part` of token n of frame tf
  auto store_rows = [&](int part, int tf, int n, long long k, const float (&y)[U][V]) {
    const __amdgpu_buffer_rsrc_t ores =
        make_rsrc_uniform(static_cast<Out*>(f.out_tokens) + size_t(k) * f.C, uint32_t(f.C) * sizeof(Out));
    const int vb = part * vpp, ve = min(nvec, vb + vpp);
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int v = vb + u * kWave + lane;
      if (v < ve) store_row<Out, V>(ores, v * V * int(sizeof(Out)), y[u]);
    }
    if (part == 0 && lane == 0) f.out_index[k] = tf * N + n;
  };
  auto store_item = [&](int j, int n, long long k, const float (&y)[U][V]) { store_rows(j % parts, t, n, k, y); };

  // s_ext[t] = kept tokens of rank >= kp in frames before t (one wave; the
  // budgets are in s_nb)
  auto fused_budget = [&]() {
    // (slots per lane for the frames at hand: the positions' layout and the
    // sums do not depend on the slot count, so neither do the budgets)
    if (T <= kWave) budget_wave_compute(bd, br, T, N, f.B, f.levels, f.tau, s_nb, s_off, nullptr);
    else if (T <= 2 * kWave) budget_wave_slots<2 * kWave>(f.rel, f.delta, T, N, f.B, f.levels, f.tau, s_nb, s_off, nullptr);
    else budget_wave_slots<kFusedTMax>(f.rel, f.delta, T, N, f.B, f.levels, f.tau, s_nb, s_off, nullptr);
  };
  auto extra_prefix = [&]() {
    int carry = 0;
    for (int t0 = 0; t0 < T; t0 += kWave) {
      const int tt = t0 + lane;
      const int e = tt < T ? max(0, s_nb[tt] - kp) : 0;
      const int incl = wave_incl_scan_i32(e);
      if (tt < T) s_ext[tt + 1] = carry + incl;
      carry += __builtin_amdgcn_readlane(incl, kWave - 1);
    }
    if (lane == 0) s_ext[0] = 0;
  };

  // read-ahead item of this wave (waves G0.., item wave - G0): its block and
  // gate are read and the row formed while the budgets are computed
  const int jp = wave - G0;
  const bool ahead = given && wave >= G0 && jp < npre;
  int np = 0;
  float yp[U][V];
  if (given) {
    if (wave >= G0) {
      u32x4 xp[U][4];
      float gp = 0.f;
      if (ahead) {
        np = f.byrank[size_t(t) * N + p + f.P * (jp / parts)];
        load_item(jp, np, xp);
        gp = f.gate[size_t(t) * N + np];
      }
      for (int n = tid - G0 * kWave; n < N; n += GW * kWave) {
        rl.rank[n] = f.rank[size_t(t) * N + n];
        rl.byrank[n] = f.byrank[size_t(t) * N + n];
        rl.gate[n] = f.gate[size_t(t) * N + n];
        if (L2) rl.gate2[n] = f.gate2[size_t(t) * N + n];
      }
      if (ahead) modulate(xp, gp, yp);
    } else {
      fused_budget();
      extra_prefix();
    }
  } else {
    // the frame's order from its scores, all waves (after the budgets)
    if constexpr (MODE == kWaveBudget) {
      if (wave == 0) fused_budget();
    }
    const __amdgpu_buffer_rsrc_t ares = make_rsrc(f.tok_score + size_t(t) * N, uint32_t(N) * 4);
    float lo = INFINITY, hi = -INFINITY;
    for (int n0 = 0; n0 < N; n0 += 4 * kThreads) {
      float av[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int n = n0 + u * kThreads + tid;
        av[u] = buf_load_f32(ares, n < N ? n * 4 : kOOB);
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int n = n0 + u * kThreads + tid;
        if (n < N) {
          rl.key[n] = sel_key(av[u], n);
          lo = fminf(lo, av[u]);
          hi = fmaxf(hi, av[u]);
        }
      }
    }
    rank_frame<kThreads>(N, f.H, f.W, f.lam, lo, hi, rl);
  }
  // LDS-only barriers from here on: the block reads stay in flight
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
  const int mine = nt > p ? (nt - p + f.P - 1) / f.P : 0;  // kept tokens of this workgroup
  const int nitems = mine * parts;

  // Output cell k of frame te under the budget-guided interpolation (Psi of
  // Eq. (17)): the grid, sample point and taps in exact integer arithmetic,
  // each tap the modulated token mu + g (x - mu) of its own 2x2 block, the
  // four blended as (1 - fy) ((1 - fx) A + fx B) + fy ((1 - fx) C + fx D).
  auto interp_item = [&](int te, int nte, int k, int part, long long row, bool own) {
    long long h0 = 1;  // the integer nearest sqrt(n H / W), halves up, within [1, H]
    while (h0 < f.H && (2 * h0 + 1) * (2 * h0 + 1) * f.W <= 4LL * nte * f.H) ++h0;
    const int gw = min(f.W, int((nte + h0 - 1) / h0)), gh = (nte + gw - 1) / gw;
    const int ci = k / gw, cj = k - ci * gw;
    auto axis = [](int i, int L, int l, int& i0, int& i1, float& fr, int& nearest) {
      const int num = (2 * i + 1) * L - l, den = 2 * l;
      i0 = num < 0 ? 0 : num / den;
      fr = num < 0 ? 0.f : float(num - i0 * den) / float(den);
      i1 = min(i0 + 1, L - 1);
      nearest = min(L - 1, ((2 * i + 1) * L) / den);
    };
    int y0, y1, ny, x0, x1, nx;
    float fy, fx;
    axis(ci, f.H, gh, y0, y1, fy, ny);
    axis(cj, f.W, gw, x0, x1, fx, nx);
    const int tap[4] = {y0 * f.W + x0, y0 * f.W + x1, y1 * f.W + x0, y1 * f.W + x1};
    const size_t fo = size_t(te) * N;
    const __amdgpu_buffer_rsrc_t xr = own ? xres : make_rsrc(static_cast<const In*>(f.X) + fo * f.C, uint32_t(N) * rb);
    u32x4 xt[4][U][4];
    float g[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      load_rows(xr, part, tap[q], xt[q]);
      g[q] = own ? rl.gate[tap[q]] : f.gate[fo + tap[q]];
    }
    float a[U][V], b[U][V], c[U][V], d[U][V], y[U][V];
    modulate(xt[0], g[0], a);
    modulate(xt[1], g[1], b);
    modulate(xt[2], g[2], c);
    modulate(xt[3], g[3], d);
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int e = 0; e < V; ++e) {
        const float top = (1.f - fx) * a[u][e] + fx * b[u][e];
        const float bottom = (1.f - fx) * c[u][e] + fx * d[u][e];
        y[u][e] = (1.f - fy) * top + fy * bottom;
      }
    store_rows(part, te, ny * f.W + nx, row, y);
  };

  // ---- B. the rows: the read-ahead one (if its token is kept), then the
  // rest, the next item's block reads in flight while one is finished ----
  auto item_token = [&](int j) { return rl.byrank[p + f.P * (j / parts)]; };
  if constexpr (INTERP) {
    if (MODE == kOffsets || !given) {
      // this workgroup's cells k = p, p + P, ... of its own frame
      for (int j = wave; j < nitems; j += kNW) {
        const int k = p + f.P * (j / parts);
        if (base + k >= 0 && base + k < total) interp_item(t, nt, k, j % parts, base + k, true);
      }
    } else {
      // every frame's cells shared out evenly over all T * P workgroups
      const long long items = (long long)s_off[T] * parts, groups = (long long)T * f.P, g = (long long)t * f.P + p;
      const long long i1 = (g + 1) * items / groups;
      for (long long i = g * items / groups + wave; i < i1; i += kNW) {
        const long long e = i / parts;
        int lo = 0, hi = T;  // s_off[lo] <= e < s_off[hi]
        while (hi - lo > 1) {
          const int mid = (lo + hi) >> 1;
          if (s_off[mid] <= e) lo = mid;
          else hi = mid;
        }
        interp_item(lo, s_off[lo + 1] - s_off[lo], int(e - s_off[lo]), int(i - e * parts), e, lo == t);
      }
    }
    return;
  }
  if (ahead && jp < nitems) {
    const long long k = base + position(np, nt);
    if (k >= 0 && k < total) store_item(jp, np, k, yp);
  }
  if constexpr (L2) {
    if (MODE == kOffsets || !given) {
      // offsets given: this workgroup's kept tokens of its frame
      for (int j = wave; j < nitems; j += kNW) {
        const int n = item_token(j);
        const long long k = base + position(n, nt);
        if (k >= 0 && k < total) {
          u32x4 x4[4][U][4];
          float y[U][V];
          load_rows2(xres, j % parts, n, x4);
          modulate2(x4, rl.gate[n], rl.gate2[n], y);
          store_item(j, n, k, y);
        }
      }
      return;
    }
  }
  if (MODE == kOffsets || !given) {
    // offsets given: this workgroup's other kept tokens of its frame
    u32x4 xa[U][4];
    int j = npre + wave;
    if (j < nitems) load_item(j, item_token(j), xa);
    for (; j < nitems; j += kNW) {
      u32x4 xb[U][4];
      const int jn = j + kNW;
      if (jn < nitems) load_item(jn, item_token(jn), xb);
      const int n = item_token(j);
      const long long k = base + position(n, nt);
      if (k >= 0 && k < total) {
        float y[U][V];
        modulate(xa, rl.gate[n], y);
        store_item(j, n, k, y);
      }
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int q = 0; q < 4; ++q) xa[u][q] = xb[u][q];
    }
    return;
  }
  // Kept tokens of rank >= kp of every frame, in (frame, rank) order and
  // split into channel parts, are shared out evenly over all T * P
  // workgroups, whatever the frames' budgets: item i of this workgroup's
  // share is token e = i / parts of that list (frame te, rank kp + e -
  // s_ext[te]), part i % parts.  Its token, gate and the frame's ranks come
  // from the per-frame kernel's arrays.
  const long long items = (long long)s_ext[T] * parts, groups = (long long)T * f.P, g = (long long)t * f.P + p;
  const long long i1 = (g + 1) * items / groups;
  for (long long i = g * items / groups + wave; i < i1; i += kNW) {
    const long long e = i / parts;
    const int part = int(i - e * parts);
    int lo = 0, hi = T;  // s_ext[lo] <= e < s_ext[hi]
    while (hi - lo > 1) {
      const int mid = (lo + hi) >> 1;
      if (s_ext[mid] <= e) lo = mid;
      else hi = mid;
    }
    const int te = lo, nte = s_nb[te], rank = kp + int(e - s_ext[te]);
    u32x4 x[L2 ? 1 : U][4], x4[L2 ? 4 : 1][L2 ? U : 1][4];
    int n, before = 0;
    float gn, gn2 = 0.f;
    if (te == t) {  // this workgroup's own frame: its order is in LDS
      n = rl.byrank[rank];
      if constexpr (L2) {
        load_rows2(xres, part, n, x4);
        gn2 = rl.gate2[n];
      } else {
        load_item(part, n, x);
      }
      gn = rl.gate[n];
      before = position(n, nte);
    } else {
      const size_t fo = size_t(te) * N;
      n = f.byrank[fo + rank];
      const __amdgpu_buffer_rsrc_t xr = make_rsrc(static_cast<const In*>(f.X) + fo * f.C, uint32_t(N) * rb);
      if constexpr (L2) {
        load_rows2(xr, part, n, x4);
        gn2 = f.gate2[fo + n];
      } else {
        load_rows(xr, part, n, x);
      }
      gn = f.gate[fo + n];
      // kept tokens of frame te before n in raster order
      const __amdgpu_buffer_rsrc_t rres = make_rsrc(f.rank + fo, uint32_t(N) * 4);
      for (int m0 = 0; m0 < n; m0 += 4 * kWave) {
        int rv[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int m = m0 + u * kWave + lane;
          rv[u] = buf_load_i32(rres, m < n ? m * 4 : kOOB);
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) before += __popcll(__ballot(m0 + u * kWave + lane < n && rv[u] < nte));
      }
    }
    const long long k = (long long)s_off[te] + before;
    if (k < total) {
      float y[U][V];
      if constexpr (L2) modulate2(x4, gn, gn2, y);
      else modulate(x, gn, y);
      store_rows(part, te, n, k, y);
    }
  }
}

template <typename In, typename Out, int MODE>
void launch_typed(const wz_config& c, const VideoArgs<AssignArgs>& a, int V, hipStream_t s) {
  const int nvec = c.C / Vec16<In>::kV;
  const dim3 grid(unsigned((c.T + kXcds - 1) / kXcds * kXcds * a.v[0].P), V), block(kThreads);
  // key 8 B; rank, byrank, gate, order / position (and level-2 gate) 4 B
  const size_t lds = size_t(c.H) * c.W * (c.spatial_levels == 2 ? 28 : 24);
  // one batch of loads per part: two vectors per lane, or one for short rows;
  // the interpolation and the two-level modulator read four blocks at once,
  // one vector per lane each
  if (c.assign == WZ_INTERP)
    hipLaunchKernelGGL((k_assign_gather<In, Out, 1, MODE, kInterp>), grid, block, lds, s, a);
  else if (c.spatial_levels == 2)
    hipLaunchKernelGGL((k_assign_gather<In, Out, 1, MODE, kSelect2>), grid, block, lds, s, a);
  else if (nvec <= kWave) hipLaunchKernelGGL((k_assign_gather<In, Out, 1, MODE, kSelect1>), grid, block, lds, s, a);
  else hipLaunchKernelGGL((k_assign_gather<In, Out, kVecPerLane, MODE, kSelect1>), grid, block, lds, s, a);
}

template <int MODE>
void launch_mode(const wz_config& c, const VideoArgs<AssignArgs>& a, int V, hipStream_t s) {
  if (c.in_dtype == WZ_BF16) {
    if (c.out_dtype == WZ_BF16) launch_typed<uint16_t, uint16_t, MODE>(c, a, V, s);
    else launch_typed<uint16_t, float, MODE>(c, a, V, s);
  } else {
    if (c.out_dtype == WZ_BF16) launch_typed<float, uint16_t, MODE>(c, a, V, s);
    else launch_typed<float, float, MODE>(c, a, V, s);
  }
}

}  // namespace

int assign_groups_per_frame(const wz_config& c, int V) {
  // about one workgroup per CU over the whole grid (all V videos), at most 16
  // per frame;
  // each repeats its frame's ranking (N^2 key comparisons), so large frames
  // get fewer
  const int tr = (c.T + kXcds - 1) / kXcds * kXcds;
  const int cap = std::max(1, std::min(16, 8192 / (c.H * c.W)));
  return std::max(1, std::min(cap, (kCUs + tr * V - 1) / (tr * V)));
}

hipError_t launch_assign_gather(const wz_config& c, const void* X, const float* tok_score, const float* frame_rel,
                                const float* frame_delta, const int32_t* offset_in, const Workspace* ws,
                                int32_t* budget_out, int32_t* offset_out, void* out_tokens, int32_t* out_index,
                                hipStream_t s, const Videos& vs) {
  // three quarters of the mean budget: most frames keep at least that many
  const int kpre = int(std::min<long long>(c.H * c.W, 3 * c.B / (4LL * c.T)));
  VideoArgs<AssignArgs> va{};
  for (int v = 0; v < vs.V; ++v) {
    AssignArgs& a = va.v[v];
    const long long w = v * vs.ws;
    a.X = advance(X, v * vs.x);
    a.tok_score = advance(tok_score, w);
    a.rel = advance(frame_rel, w);
    a.delta = advance(frame_delta, w);
    a.offset_in = advance(offset_in, v * vs.off);
    a.rank = ws ? advance(ws->rank, w) : nullptr;
    a.byrank = ws ? advance(ws->byrank, w) : nullptr;
    a.gate = ws ? advance(ws->gate, w) : nullptr;
    a.gate2 = ws ? advance(ws->gate2, w) : nullptr;
    a.budget_out = advance(budget_out, v * vs.bud);
    a.offset_out = advance(offset_out, v * vs.off);
    a.out_tokens = advance(out_tokens, v * vs.out);
    a.out_index = advance(out_index, v * vs.idx);
    a.B = c.B;
    a.T = c.T;
    a.H = c.H;
    a.W = c.W;
    a.C = c.C;
    a.P = assign_groups_per_frame(c, vs.V);
    a.levels = c.levels;
    a.kpre = kpre;
    a.lam = c.lambda_;
    a.tau = c.tau;
  }
  if (offset_in) launch_mode<kOffsets>(c, va, vs.V, s);
  else if (c.T <= kFusedTMax) launch_mode<kWaveBudget>(c, va, vs.V, s);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace wz
