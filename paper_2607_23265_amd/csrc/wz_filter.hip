// Stage 3 with a db4 or bior4.4 spatial basis: the Wavelet Spatial Modulator
// of Eq. (12)-(15) with a filter bank (wz_wavelets.h), the selection that
// replaces Eq. (17) and the compaction of Eq. (19).
//
// One level of the separable 2-D transform, its three detail bands
// multiplied by G = lambda * P(M) (Eq. (13)-(14), P the adaptive average
// pooling of the frame's saliency map M (Eq. (7)) to the n_h x n_w subband
// grid) and the inverse (Eq. (15)) is a linear map of each channel's H x W
// map.  Written per axis with analysis rows a_u[i][.] and synthesis weights
// s_u[h][i] = rec_u[h + F - 2 - 2i] (u = lo, hi), the reconstructed token
// p = (h, w) is
//   x~_p = sum_{h', w'} L_p(h', w') x_{h', w'},
//   L_p(h', w') = sum_{i, j} (1 - G_ij) E_i(h') E'_j(w') + G_ij P_i(h') P'_j(w'),
// with E_i(h') = s_lo[h][i] a_lo[i][h'] (the approximation path along the
// height) and P_i(h') = E_i(h') + s_hi[h][i] a_hi[i][h'] (both paths), E' and
// P' likewise along the width: the approximation band LL passes unchanged and
// the three detail bands get G.  Only i with s_u[h][i] != 0 contribute (at
// most F / 2 of them), j likewise.
//
// Fused form, workgroup (frame t, channel slice), 512 threads (eight waves
// share the slice-independent setup, which every slice's workgroup repeats):
//   1. takes the frame's selection ranks (from the per-frame kernel, or forms
//      them from the scores, wz_rank.h) and lists its n_t kept tokens
//      (rank < n_t) in raster order.  With the whole pass, T <= 64 and the
//      Haar temporal basis, wave 0 first computes every frame's budget
//      (Eq. (9)-(11), Eq. (16) under Eq. (5); the selection kernel's one-wave
//      arithmetic, so every workgroup gets the same budgets bit for bit)
//      while the other waves read the ranks, and no budget launch precedes
//      this one;
//   2. forms G and the per-axis analysis rows a_u in LDS;
//   3. per chunk of KR kept tokens builds their rows L_p in LDS (fp32,
//      through the partial sums B_i(w') = sum_j over the width) and
//      contracts them with the frame's slice, a dense product of KR rows,
//      H*W tokens and the slice's channels: for bf16 inputs on MFMA (the rows
//      split into bf16 high and low parts, fp32 accumulation; each wave takes
//      128 channels of a 1024-channel slice), for fp32 inputs on the vector
//      ALU (512-channel slices, each wave an eighth of the rows, fp32); then
//      writes the rows to
//      out_tokens[offset_t + k] (k = raster position among the kept tokens),
//      their flat indices to out_index.
// The frame's slice is read once per chunk of KR kept tokens (from L2 after
// the first, while the slices of the workgroups on an XCD fit its L2).
// Split form (bf16 inputs on frames where LDS holds full-frame rows for at
// most 16 kept tokens, which would read the slice from memory once per
// chunk): the same kernel with ROWS, one workgroup per frame, does 1-3 and
// writes the rows to the workspace instead of contracting them; then
// k_filter_contract keeps up to 48 rows in its accumulators while each wave
// streams its 128 channels of the frame once.
// Supported: H, W <= 64, H*W <= 1024 (the host checks).
#include "wz_budget.h"
#include "wz_rank.h"
#include "wz_wavelets.h"

namespace wz {
namespace {

constexpr int kFThreads = 512;
constexpr int kFWaves = kFThreads / kWave;
// channels of a workgroup: 128 per wave on MFMA (bf16 inputs); 8 per lane on
// the vector ALU (fp32 inputs), where the waves split the rows instead
constexpr int kFSliceMf = kFWaves * 128;
constexpr int kFSliceValu = kWave * 8;
constexpr int filter_slice(bool mfma) { return mfma ? kFSliceMf : kFSliceValu; }
constexpr int kMaxAct = kMaxTaps / 2;  // synthesis rows touching one output sample

struct FilterArgs {
  const void* X;            // [T][H][W][C]
  const float* tok_score;   // [T][H*W]
  const int32_t* offset;    // [T+1], or null: the budgets are computed here
  const float* rel;         // [T] r_t        (budgets computed here; T <= 64, Haar temporal basis)
  const float* delta;       // [T] delta_t
  int32_t* budget_out;      // [T] or null    (budgets computed here; written by workgroup (0, 0))
  int32_t* offset_out;      // [T+1]          (budgets computed here)
  const int32_t* rank;      // [T][H*W] selection ranks from the per-frame kernel, or null (ranked here)
  uint16_t* rows;           // [B][2][pad_tokens(H*W)] the row kernel's output (bf16 high, low part)
  void* out_tokens;         // [B][C]
  int32_t* out_index;       // [B]
  long long B;
  int T, H, W, C, levels;
  float lam, tau;
};
static_assert(sizeof(VideoArgs<FilterArgs>) <= 4096, "per-video arguments exceed the kernel argument limit");

// 8 channels of a token row: raw 16-byte vectors (one for bf16, two for
// fp32) and their widening to floats.
template <typename In>
struct Raw8 {
  static constexpr int kV = sizeof(In) == 2 ? 1 : 2;
  u32x4 v[kV];
  __device__ __forceinline__ void load(__amdgpu_buffer_rsrc_t r, int off) {
#pragma unroll
    for (int i = 0; i < kV; ++i) v[i] = __builtin_amdgcn_raw_buffer_load_b128(r, off + 16 * i, 0, 0);
  }
  __device__ __forceinline__ void widen(float (&x)[8]) const {
    if constexpr (kV == 1) {
#pragma unroll
      for (int i = 0; i < 4; ++i) { x[2 * i] = bf16_lo(v[0][i]); x[2 * i + 1] = bf16_hi(v[0][i]); }
    } else {
#pragma unroll
      for (int i = 0; i < 4; ++i) { x[i] = __uint_as_float(v[0][i]); x[4 + i] = __uint_as_float(v[1][i]); }
    }
  }
};
template <typename Out>
__device__ __forceinline__ void store8(__amdgpu_buffer_rsrc_t r, int off, const float (&v)[8]);
template <>
__device__ __forceinline__ void store8<uint16_t>(__amdgpu_buffer_rsrc_t r, int off, const float (&v)[8]) {
  u32x4 o;
#pragma unroll
  for (int i = 0; i < 4; ++i) o[i] = f32_to_bf16_rne(v[2 * i]) | (f32_to_bf16_rne(v[2 * i + 1]) << 16);
  buf_store_wt_b128(o, r, off);
}
template <>
__device__ __forceinline__ void store8<float>(__amdgpu_buffer_rsrc_t r, int off, const float (&v)[8]) {
  buf_store_wt_b128(u32x4{__float_as_uint(v[0]), __float_as_uint(v[1]), __float_as_uint(v[2]), __float_as_uint(v[3])},
                    r, off);
  buf_store_wt_b128(u32x4{__float_as_uint(v[4]), __float_as_uint(v[5]), __float_as_uint(v[6]), __float_as_uint(v[7])},
                    r, off + 16);
}

// Dynamic LDS of a frame of H x W tokens and chunks of kr rows: byte offsets
// of the arrays (the operator rows 16-byte aligned) and the total.
struct FilterLds {
  size_t M, kept, G, AH, AW, SH, SW, B, L, det, bytes;
};
// Tokens padded to whole MFMA K steps, and the row stride (bf16 elements) of
// the operator rows in their MFMA form: 8 more than the padded length, so the
// 16 rows that 16 lanes read at once fall in distinct LDS banks.
__host__ __device__ inline int pad_tokens(int N) { return (N + 31) / 32 * 32; }
__host__ __device__ inline int mfma_row_stride(int N) { return pad_tokens(N) + 8; }
// mfma: the operator rows as bf16 high and low parts
// [2][max(kr, 16)][mfma_row_stride] (bf16 inputs; whole 16-row MFMA tiles)
// instead of fp32 [N][kr].  det_levels: the budget's detail coefficients
// [det_levels][kWave] fp64 last (budgets computed in the kernel), or none.
__host__ __device__ inline FilterLds filter_lds(int H, int W, int F, int kr, bool mfma, int det_levels = 0) {
  const size_t N = size_t(H) * W, nh = bank_len(H, F), nw = bank_len(W, F);
  FilterLds o;
  // the ranking's key, rank, byrank, gate and bin order come first (24 N bytes)
  o.M = N * 24;                               // saliency M [N]
  o.kept = o.M + N * 4;                       // kept tokens in raster order [N]
  o.G = o.kept + N * 4;                       // gates [nh][nw]
  o.AH = o.G + nh * nw * 4;                   // analysis rows along the height [2][nh][H]
  o.AW = o.AH + 2 * nh * H * 4;               // along the width [2][nw][W]
  o.SH = o.AW + 2 * nw * W * 4;               // synthesis weights along the height [2][H][kMaxAct]
  o.SW = o.SH + 2 * size_t(H) * kMaxAct * 4;  // along the width [2][W][kMaxAct]
  o.B = o.SW + 2 * size_t(W) * kMaxAct * 4;   // partial sums B1, B2 [kr][2][kMaxAct][W]
  o.L = (o.B + size_t(kr) * 2 * kMaxAct * W * 4 + 15) / 16 * 16;  // operator rows [N][kr], 16-byte aligned
  o.det = o.L + (mfma ? size_t(2) * (kr < 16 ? 16 : kr) * mfma_row_stride(int(N)) * 2 : N * kr * 4);
  o.bytes = o.det + size_t(det_levels) * kWave * 8;
  return o;
}

// The contraction of R operator rows with the frame's slice: a ring of D
// token rows in flight per wave (16-byte vectors of 8 channels per lane),
// fp32 accumulation, then the rows written to out_tokens (and, by slice 0,
// their flat indices).
struct ContractArgs {
  __amdgpu_buffer_rsrc_t xres;
  int xoff, rb, N, KR;
  const float* L;  // the first row's column of the operator rows [N][KR]
  int k0, nt;      // the first row's raster position; the frame's kept tokens
  long long base, total;
  int C;
  bool vok;
  int v, sl, lane, t;
  const int32_t* kept;
  void* out_tokens;
  int32_t* out_index;
};
template <typename In, typename Out, int R>
__device__ __forceinline__ void contract_rows(const ContractArgs& a) {
  float acc[R][8];
#pragma unroll
  for (int r = 0; r < R; ++r)
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[r][e] = 0.f;
  constexpr int D = 16;
  Raw8<In> ring[D];
#pragma unroll
  for (int d = 0; d < D; ++d) ring[d].load(a.xres, d < a.N ? d * a.rb + a.xoff : kOOB);
  for (int n0 = 0; n0 < a.N; n0 += D) {
#pragma unroll
    for (int d = 0; d < D; ++d) {
      const int n = n0 + d;
      float xc[8];
      ring[d].widen(xc);
      ring[d].load(a.xres, n + D < a.N ? (n + D) * a.rb + a.xoff : kOOB);
      if (n < a.N) {
        const float* Ln = a.L + n * a.KR;
#pragma unroll
        for (int r = 0; r < R; ++r) {
          const float l = Ln[r];
#pragma unroll
          for (int e = 0; e < 8; ++e) acc[r][e] = fmaf(l, xc[e], acc[r][e]);
        }
      }
    }
  }
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int k = a.k0 + r;
    if (k < a.nt && a.base + k < a.total) {
      const __amdgpu_buffer_rsrc_t ores = make_rsrc_uniform(
          static_cast<Out*>(a.out_tokens) + size_t(a.base + k) * a.C, uint32_t(a.C) * sizeof(Out));
      if (a.vok) store8<Out>(ores, a.v * 8 * int(sizeof(Out)), acc[r]);
      if (a.sl == 0 && a.lane == 0) a.out_index[a.base + k] = a.t * (a.N) + a.kept[k];
    }
  }
}

// ROWS (bf16 inputs): the row kernel of the split form, one workgroup per
// frame: steps 1-3b, then the chunk's operator rows (MFMA form) go to
// f.rows and their flat indices to out_index, for k_filter_contract.
template <typename In, typename Out, int KR, bool ROWS = false>
__global__ __launch_bounds__(kFThreads) void k_filter_assign(const VideoArgs<FilterArgs> va, const Bank bank) {
  constexpr int RW = KR / kFWaves;  // rows a wave contracts
  const FilterArgs& f = va.v[blockIdx.y];
  constexpr int SLICE = filter_slice(sizeof(In) == 2);
  const int S = ROWS ? 1 : (f.C + SLICE - 1) / SLICE;
  const int b = blockIdx.x, xcd = b % kXcds, slot = b / kXcds;
  const int t = (slot / S) * kXcds + xcd, sl = slot % S;
  if (t >= f.T) return;  // whole workgroup
  const int H = f.H, W = f.W, N = H * W, F = bank.F, C = f.C;
  const int nh = bank_len(H, F), nw = bank_len(W, F);
  // with the offsets given, a frame that keeps nothing is done; otherwise
  // wave 0 computes the budgets (from r and delta, the selection kernel's
  // one-wave arithmetic) while the other waves take the frame's ranks and
  // build the tables
  const bool wb = f.offset == nullptr;
  long long base = 0, total = 0;
  int nt = 0;
  if (!wb) {
    base = f.offset[t];
    nt = min(max(f.offset[t + 1] - int(base), 0), N);
    total = min((long long)f.offset[f.T], f.B);
    if (nt == 0) return;  // whole workgroup
  }
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  // threads that rank and build while wave 0 computes the budgets
  const int g0 = wb ? kWave : 0, gtid = tid - g0, gthreads = kFThreads - g0;

  extern __shared__ __align__(16) char s_dyn[];
  __shared__ int s_start[kBins], s_fill[kBins];
  __shared__ float s_mm[2 * kFWaves];
  __shared__ int s_wsum[kFWaves];
  __shared__ int32_t s_nb[kWave], s_off[kWave + 1];  // budgets and offsets (computed here)
  RankLds rl;
  rl.key = reinterpret_cast<uint64_t*>(s_dyn);
  rl.rank = reinterpret_cast<int32_t*>(rl.key + N);
  rl.byrank = rl.rank + N;
  rl.gate = reinterpret_cast<float*>(rl.byrank + N);
  rl.order = reinterpret_cast<int32_t*>(rl.gate + N);
  rl.gate2 = nullptr;
  rl.start = s_start;
  rl.fill = s_fill;
  rl.mm = s_mm;
  constexpr bool MF = sizeof(In) == 2;  // bf16 inputs: the contraction runs on MFMA
  const FilterLds lo_ = filter_lds(H, W, F, KR, MF, wb ? f.levels : 0);
  float* s_M = reinterpret_cast<float*>(s_dyn + lo_.M);           // [N] saliency M
  int32_t* s_kept = reinterpret_cast<int32_t*>(s_dyn + lo_.kept);  // [nt] kept tokens in raster order
  float* s_G = reinterpret_cast<float*>(s_dyn + lo_.G);           // [nh][nw] gates
  float* s_AH = reinterpret_cast<float*>(s_dyn + lo_.AH);         // [2][nh][H] analysis rows along the height
  float* s_AW = reinterpret_cast<float*>(s_dyn + lo_.AW);         // [2][nw][W] along the width
  float* s_SH = reinterpret_cast<float*>(s_dyn + lo_.SH);         // [2][H][kMaxAct] synthesis weights
  float* s_SW = reinterpret_cast<float*>(s_dyn + lo_.SW);         // [2][W][kMaxAct]
  float* s_B = reinterpret_cast<float*>(s_dyn + lo_.B);           // [KR][2][kMaxAct][W]
  float* s_L = reinterpret_cast<float*>(s_dyn + lo_.L);           // [N][KR] operator rows, token-major
  uint16_t* s_Lh = reinterpret_cast<uint16_t*>(s_dyn + lo_.L);    // MFMA form: [2][LR][LS] bf16 high, low
  constexpr int LR = KR < 16 ? 16 : KR;                            // rows of a part: whole 16-row tiles
  const int LS = mfma_row_stride(N), NP = pad_tokens(N);

  // ---- 1. ranks from the scores (and the budgets); kept tokens in raster order ----
  if (wb && wave == 0) {
    const double d = lane < f.T ? double(f.delta[lane]) : 0.0, r = lane < f.T ? double(f.rel[lane]) : 0.0;
    budget_wave_compute_det(d, r, f.T, N, f.B, f.levels, f.tau, s_nb, s_off, nullptr,
                            reinterpret_cast<double*>(s_dyn + lo_.det));
    if (lane == 0) {  // no scores in this wave
      s_mm[0] = INFINITY;
      s_mm[kFWaves] = -INFINITY;
    }
  } else {
    const __amdgpu_buffer_rsrc_t ares = make_rsrc(f.tok_score + size_t(t) * N, uint32_t(N) * 4);
    float lo = INFINITY, hi = -INFINITY;
    for (int n0 = 0; n0 < N; n0 += 4 * gthreads) {
      float av[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int n = n0 + u * gthreads + gtid;
        av[u] = buf_load_f32(ares, n < N ? n * 4 : kOOB);
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int n = n0 + u * gthreads + gtid;
        if (n < N) {
          rl.key[n] = sel_key(av[u], n);
          lo = fminf(lo, av[u]);
          hi = fmaxf(hi, av[u]);
        }
      }
    }
    if (f.rank) {
      // the per-frame kernel's ranks (the same ranking of the same keys); the
      // frame's score extremes per wave, as the ranking leaves them
      for (int n = gtid; n < N; n += gthreads) rl.rank[n] = f.rank[size_t(t) * N + n];
      lo = wave_min_f32(lo);
      hi = wave_max_f32(hi);
      if (lane == 0) {
        s_mm[wave] = lo;
        s_mm[kFWaves + wave] = hi;
      }
    } else {
      // (the offsets are given whenever the ranks are not, so every wave is here)
      rank_frame<kFThreads>(N, H, W, f.lam, lo, hi, rl);
    }
  }
  __syncthreads();
  if (wb) {
    base = s_off[t];
    nt = min(s_off[t + 1] - s_off[t], N);
    total = min((long long)s_off[f.T], f.B);
    if (t == 0 && sl == 0) {
      for (int i = tid; i <= f.T; i += kFThreads) {
        if (i < f.T && f.budget_out) f.budget_out[i] = s_nb[i];
        f.offset_out[i] = s_off[i];
      }
    }
    if (nt == 0) return;  // whole workgroup
  }
  {
    // the frame's extremes, as the ranking formed them; M by Eq. (7)
    float lo = s_mm[0], hi = s_mm[kFWaves];
#pragma unroll
    for (int w = 1; w < kFWaves; ++w) {
      lo = fminf(lo, s_mm[w]);
      hi = fmaxf(hi, s_mm[kFWaves + w]);
    }
    const float range = hi - lo;
    for (int n = tid; n < N; n += kFThreads) {
      const float a = order_value(uint32_t(rl.key[n] >> 12));
      s_M[n] = range > 0.f ? (a - lo) / range : 0.f;
    }
    // kept list: thread tid takes tokens 4 tid .. 4 tid + 3 (N <= 1024)
    int flag[4], cnt = 0;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int n = 4 * tid + e;
      flag[e] = n < N && rl.rank[n] < nt;
      cnt += flag[e];
    }
    const int incl = wave_incl_scan_i32(cnt);
    if (lane == kWave - 1) s_wsum[wave] = incl;
    __syncthreads();
    int pos = incl - cnt;
    for (int w = 0; w < wave; ++w) pos += s_wsum[w];
#pragma unroll
    for (int e = 0; e < 4; ++e)
      if (flag[e]) s_kept[pos++] = 4 * tid + e;
  }
  __syncthreads();

  // ---- 2. gates G = lambda * (mean of M over each subband cell's bins) and
  // the analysis rows a_u[i][.] of both axes ----
  for (int q = tid; q < nh * nw; q += kFThreads) {
    const int i = q / nw, j = q - i * nw;
    const int h0 = (i * H) / nh, h1 = ((i + 1) * H + nh - 1) / nh;
    const int w0 = (j * W) / nw, w1 = ((j + 1) * W + nw - 1) / nw;
    float s = 0.f;
    for (int h = h0; h < h1; ++h)
      for (int w = w0; w < w1; ++w) s += s_M[h * W + w];
    s_G[q] = f.lam * (s / float((h1 - h0) * (w1 - w0)));
  }
  for (int q = tid; q < 2 * nh + 2 * nw; q += kFThreads) {
    // one row per thread: band u of index i along an axis of length len
    const bool height = q < 2 * nh;
    const int r = height ? q : q - 2 * nh, n = height ? nh : nw, len = height ? H : W;
    const int u = r / n, i = r - u * n;
    float* row = (height ? s_AH : s_AW) + (u * n + i) * len;
    for (int x = 0; x < len; ++x) row[x] = 0.f;
    for (int j = 0; j < F; ++j) row[sym_index(2 * i + 1 - j, len)] += float(u == 0 ? bank.dec_lo[j] : bank.dec_hi[j]);
  }
  // synthesis weights: coefficient i = x / 2 + ii (the first of at most
  // kMaxAct whose filter reaches x) of band u at output position x,
  // rec_u[x + F - 2 - 2i], 0 outside the filter or past the band
  for (int q = tid; q < 2 * (H + W) * kMaxAct; q += kFThreads) {
    const bool height = q < 2 * H * kMaxAct;
    const int r = height ? q : q - 2 * H * kMaxAct, len = height ? H : W, n = height ? nh : nw;
    const int u = r / (len * kMaxAct), x = (r / kMaxAct) % len, ii = r % kMaxAct;
    const int i = x / 2 + ii, k = x + F - 2 - 2 * i;
    (height ? s_SH : s_SW)[r] =
        (i < n && k >= 0 && k < F) ? float(u == 0 ? bank.rec_lo[k] : bank.rec_hi[k]) : 0.f;
  }
  __syncthreads();

  if constexpr (MF && KR < LR) {  // rows KR .. 15 of each part stay zero
    for (int q = tid; q < 2 * (LR - KR) * LS; q += kFThreads) {
      const int part = q / ((LR - KR) * LS), rem = q - part * (LR - KR) * LS;
      s_Lh[(part * LR + KR) * LS + rem] = 0;
    }
  }
  const int nvec = C / 8;  // 8-channel vectors of a row
  const int v = sl * kWave + lane;
  const bool vok = v < nvec;
  const int rb = C * int(sizeof(In));
  const __amdgpu_buffer_rsrc_t xres = make_rsrc(static_cast<const In*>(f.X) + size_t(t) * N * C, uint32_t(N) * rb);
  const int xoff = vok ? v * 8 * int(sizeof(In)) : kOOB;

  for (int c0 = 0; c0 < nt; c0 += KR) {
    // ---- 3a. B1_i(w') = sum_j (1 - G_ij) E'_j(w'), B2_i(w') = sum_j G_ij P'_j(w')
    // for the chunk's rows, i over the coefficients reaching the row's h ----
    for (int q = tid; q < KR * kMaxAct * W; q += kFThreads) {
      const int r = q / (kMaxAct * W), rem = q - r * (kMaxAct * W), ii = rem / W, x = rem - ii * W;
      float b1 = 0.f, b2 = 0.f;
      if (c0 + r < nt) {
        const int p = s_kept[c0 + r], h = p / W, w = p - h * W;
        const int i = h / 2 + ii;
        if (i < nh) {
          const int j0 = w / 2;
#pragma unroll
          for (int jj = 0; jj < kMaxAct; ++jj) {
            const int j = min(j0 + jj, nw - 1);  // weights past the band are 0
            const float e = s_SW[(0 * W + w) * kMaxAct + jj] * s_AW[j * W + x];
            const float pp = e + s_SW[(1 * W + w) * kMaxAct + jj] * s_AW[(nw + j) * W + x];
            const float g = s_G[i * nw + j];
            b1 += (1.f - g) * e;
            b2 += g * pp;
          }
        }
      }
      s_B[((r * 2 + 0) * kMaxAct + ii) * W + x] = b1;
      s_B[((r * 2 + 1) * kMaxAct + ii) * W + x] = b2;
    }
    __syncthreads();
    // ---- 3b. L_p(h', w') = sum_i E_i(h') B1_i(w') + P_i(h') B2_i(w'): thread
    // tid builds row tid % KR at columns w' = tid / KR, + 512 / KR, ..., each
    // column's B values in registers and the height factors read per h' (the
    // same for all of the row's threads: one LDS broadcast) ----
    {
      const int r = tid % KR, nstep = kFThreads / KR;
      const bool live = c0 + r < nt;
      float ew[kMaxAct], pw[kMaxAct];
      int ih[kMaxAct];
      const int h = live ? s_kept[c0 + r] / W : 0;
#pragma unroll
      for (int ii = 0; ii < kMaxAct; ++ii) {
        ih[ii] = min(h / 2 + ii, nh - 1);  // weights past the band are 0
        ew[ii] = live ? s_SH[(0 * H + h) * kMaxAct + ii] : 0.f;
        pw[ii] = live ? s_SH[(1 * H + h) * kMaxAct + ii] : 0.f;
      }
      const float* B1 = s_B + (r * 2 + 0) * kMaxAct * W;
      const float* B2 = s_B + (r * 2 + 1) * kMaxAct * W;
      auto put = [&](int n, float acc) {
        if constexpr (MF) {
          // bf16 high part and the rounded remainder: together about 16
          // significant bits of the row entry (tokens past N are 0)
          const uint32_t hi = f32_to_bf16_rne(acc);
          s_Lh[r * LS + n] = uint16_t(hi);
          s_Lh[(LR + r) * LS + n] = uint16_t(f32_to_bf16_rne(acc - __uint_as_float(hi << 16)));
        } else {
          s_L[n * KR + r] = acc;
        }
      };
      for (int x = tid / KR; x < W; x += nstep) {
        float b1[kMaxAct], b2[kMaxAct];
#pragma unroll
        for (int ii = 0; ii < kMaxAct; ++ii) {
          b1[ii] = B1[ii * W + x];
          b2[ii] = B2[ii * W + x];
        }
        // two image rows at a time: the next row's LDS reads issue before this
        // one's entries are finished
#pragma unroll 2
        for (int y = 0; y < H; ++y) {
          float acc = 0.f;
#pragma unroll
          for (int ii = 0; ii < kMaxAct; ++ii) {
            const float e = ew[ii] * s_AH[ih[ii] * H + y];
            const float pp = e + pw[ii] * s_AH[(nh + ih[ii]) * H + y];
            acc += e * b1[ii] + pp * b2[ii];
          }
          put(y * W + x, acc);
        }
      }
      if constexpr (MF)
        for (int n = N + tid / KR; n < NP; n += nstep) put(n, 0.f);
    }
    __syncthreads();
    if constexpr (ROWS) {
      // ---- 3c. the chunk's rows to the row buffer (both parts, NP tokens
      // each; 16 bytes a thread) and their flat indices ----
      const int nr = min(KR, nt - c0), vr = NP / 8;
      for (int q = tid; q < nr * 2 * vr; q += kFThreads) {
        const int r = q / (2 * vr), rem = q - r * (2 * vr), part = rem / vr, v8 = rem - part * vr;
        if (base + c0 + r < total)
          *reinterpret_cast<u32x4*>(f.rows + (size_t(base + c0 + r) * 2 + part) * NP + 8 * v8) =
              *reinterpret_cast<const u32x4*>(s_Lh + (part * LR + r) * LS + 8 * v8);
      }
      for (int r = tid; r < nr; r += kFThreads)
        if (base + c0 + r < total) f.out_index[base + c0 + r] = t * N + s_kept[c0 + r];
    } else if constexpr (MF) {
    // ---- 3c. the chunk's rows against the frame's slice ----
      // MFMA: C[rows][channels] += L[rows][tokens] X[tokens][channels] with
      // v_mfma_f32_16x16x32_bf16, the wave's 128 channels in 8 MFMAs per
      // 16-row tile and 32-token step.  Lane (r16, g) = (lane % 16, lane / 16)
      // loads tokens 8g .. 8g+7 of the step for its 8 channels 8 r16 .. 8 r16+7
      // and transposes the 8 x 8 block in registers: w[c'] holds the 8 tokens
      // of channel 8 r16 + c', which is exactly the B operand (8 K values of
      // column r16) of MFMA c', whose columns are channels 8 r16 + c'.  The A
      // operand is the rows' bf16 high or low part, 8 tokens from LDS.  Lane
      // (r16, g) ends with rows 4g .. 4g+3 of each tile for its 8 consecutive
      // channels.
      const int nr = min(KR, nt - c0);
      constexpr int RT = (KR + 15) / 16;  // 16-row tiles
      const int rtiles = (nr + 15) / 16;
      const int r16 = lane & 15, g = lane >> 4;
      const int cw = sl * SLICE + wave * 128 + 8 * r16;  // the lane's first channel
      const int coff = cw < C ? cw * 2 : kOOB;
      f32x4 acc[RT][8];
#pragma unroll
      for (int i = 0; i < RT; ++i)
#pragma unroll
        for (int c = 0; c < 8; ++c) acc[i][c] = f32x4{0.f, 0.f, 0.f, 0.f};
      // tokens 8g + e of a step, channels 8 r16 .. +7; past the frame: zeros
      auto load_step = [&](int k0, u32x4 (&d)[8]) {
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int n = k0 + 8 * g + e;
          d[e] = __builtin_amdgcn_raw_buffer_load_b128(xres, (n < N && coff != kOOB) ? n * rb + coff : kOOB, 0, 0);
        }
      };
      auto step = [&](int k0, const u32x4 (&x)[8]) {
        // 8 x 8 transpose of bf16: w[c'] dword j = tokens (2j, 2j+1) of channel c'
        u32x4 w[8];
#pragma unroll
        for (int m = 0; m < 4; ++m)
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            w[2 * m][j] = __builtin_amdgcn_perm(x[2 * j + 1][m], x[2 * j][m], 0x05040100u);
            w[2 * m + 1][j] = __builtin_amdgcn_perm(x[2 * j + 1][m], x[2 * j][m], 0x07060302u);
          }
#pragma unroll
        for (int i = 0; i < RT; ++i) {
          if (i >= rtiles) break;
          const int row = 16 * i + r16;
          const bf16x8 ah = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(s_Lh + row * LS + k0 + 8 * g));
          const bf16x8 al =
              __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(s_Lh + (LR + row) * LS + k0 + 8 * g));
#pragma unroll
          for (int c = 0; c < 8; ++c) {
            const bf16x8 bw = __builtin_bit_cast(bf16x8, w[c]);
            acc[i][c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, bw, acc[i][c], 0, 0, 0);
            acc[i][c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al, bw, acc[i][c], 0, 0, 0);
          }
        }
      };
      // a two-slot ring of steps, issued in slot order and reloaded in place
      // (a register copy of a slot still loading would wait for the load): the
      // next step's block is in flight while one is contracted
      u32x4 xa[8], xb[8];
      load_step(0, xa);
      __builtin_amdgcn_sched_barrier(0);
      load_step(32, xb);
      for (int k0 = 0; k0 < NP; k0 += 64) {
        __builtin_amdgcn_sched_barrier(0);
        step(k0, xa);
        load_step(k0 + 64, xa);
        __builtin_amdgcn_sched_barrier(0);
        if (k0 + 32 < NP) step(k0 + 32, xb);
        load_step(k0 + 96, xb);
      }
#pragma unroll
      for (int i = 0; i < RT; ++i) {
        if (i >= rtiles) break;
        // one descriptor per 16-row tile (the lanes' rows differ); its size
        // stops at the last row the call may write
        const long long row0 = base + c0 + 16 * i;
        const long long rows = min(16LL, total - row0);
        const __amdgpu_buffer_rsrc_t ores = make_rsrc_uniform(
            static_cast<Out*>(f.out_tokens) + size_t(row0) * C, rows > 0 ? uint32_t(rows * C * sizeof(Out)) : 0u);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int rt = 4 * g + e, k = c0 + 16 * i + rt;
          if (k < nt && base + k < total) {
            float y8[8];
#pragma unroll
            for (int c = 0; c < 8; ++c) y8[c] = acc[i][c][e];
            if (cw < C) store8<Out>(ores, (rt * C + cw) * int(sizeof(Out)), y8);
            if (sl == 0 && wave == 0 && r16 == 0) f.out_index[base + k] = t * N + s_kept[k];
          }
        }
      }
    } else {
      // VALU (fp32 inputs): the chunk's rows spread evenly over the waves (a
      // wave with R rows runs the R-row contraction)
      const int nr = min(KR, nt - c0), rw = (nr + kFWaves - 1) / kFWaves;
      const int row0 = wave * rw, mine = max(0, min(rw, nr - row0));
      ContractArgs ca{xres, xoff, rb, N, KR, s_L + row0, c0 + row0, nt, base, total, C, vok, v, sl, lane, t,
                      s_kept, f.out_tokens, f.out_index};
      switch (mine) {
        case 1: contract_rows<In, Out, 1>(ca); break;
        case 2: contract_rows<In, Out, 2>(ca); break;
        case 3: contract_rows<In, Out, 3>(ca); break;
        case 4: contract_rows<In, Out, 4>(ca); break;
        case 5: if constexpr (RW >= 5) contract_rows<In, Out, 5>(ca); break;
        case 6: if constexpr (RW >= 6) contract_rows<In, Out, 6>(ca); break;
        case 7: if constexpr (RW >= 7) contract_rows<In, Out, 7>(ca); break;
        case 8: if constexpr (RW >= 8) contract_rows<In, Out, 8>(ca); break;
        default: break;
      }
    }
    __syncthreads();  // the next chunk rewrites B and L
  }
}

// The split form's contraction (bf16 inputs): out_tokens rows of frame t =
// its operator rows (from the row kernel) times the frame's tokens.
struct RowsArgs {
  const void* X;           // [T][H][W][C] bf16
  const int32_t* offset;   // [T+1]
  const uint16_t* rows;    // [B][2][pad_tokens(N)]
  void* out_tokens;        // [B][C]
  long long B;
  int T, N, C;
};
static_assert(sizeof(VideoArgs<RowsArgs>) <= 4096, "per-video arguments exceed the kernel argument limit");
// A frame's channels in S slices of at most four 128-channel waves, the
// slices balanced (each a multiple of 128 channels).  At the contraction's
// register use (two waves a SIMD) a CU holds eight of its waves: four-wave
// workgroups, two to a CU, keep more of them live than eight-wave ones when a
// frame's channels leave part of a workgroup without any (at C = 1152: six
// live waves a CU against four or five).
constexpr int kRcWaveCh = 128;
constexpr int kRcWaves = 4;
__host__ __device__ inline int rc_slices(int C) { return (C + kRcWaves * kRcWaveCh - 1) / (kRcWaves * kRcWaveCh); }
__host__ __device__ inline int rc_slice_width(int C, int S) {
  return ((C + S - 1) / S + kRcWaveCh - 1) / kRcWaveCh * kRcWaveCh;
}

// Workgroup (frame t, channel slice), 4 waves of 128 channels each: sweeps
// of up to 16 RT rows, whose accumulators stay in registers while each wave
// streams its 128 channels of the frame once.  The sweep's operator entries
// (the same for every wave) are staged once per workgroup through LDS in
// 128-token blocks, double-buffered: the next block's entries load while the
// block is contracted, one LDS barrier a block; a wave without channels only
// stages.  C[rows][channels] += L[rows][tokens] X[tokens][channels] with
// v_mfma_f32_16x16x32_bf16, 8 MFMAs per 16-row tile and 32-token step (each
// twice: the rows' bf16 high and low parts).  Lane (r16, g) =
// (lane % 16, lane / 16) loads tokens 8g .. 8g+7 of a step for its channels
// 8 r16 .. 8 r16+7 (16 bytes a token); the B operand of MFMA c' (8 K values
// of column r16) is channel 8 r16 + c' of those tokens, formed by byte
// permutes just before its MFMAs, so that the columns of MFMA c' are
// channels 8 r16 + c'.  The A operand (row 16i + r16, tokens 8g .. 8g+7) is
// one 16-byte LDS read per part.  Lane (r16, g) ends with rows 4g .. 4g+3 of
// each tile for its 8 consecutive channels.
template <typename Out, int RT>
__global__ __launch_bounds__(kRcWaves * kWave) __attribute__((amdgpu_waves_per_eu(2))) void k_filter_contract(const VideoArgs<RowsArgs> va) {
  const RowsArgs& f = va.v[blockIdx.y];
  const int S = rc_slices(f.C);
  const int b = blockIdx.x, xcd = b % kXcds, slot = b / kXcds;
  const int t = (slot / S) * kXcds + xcd, sl = slot % S;
  if (t >= f.T) return;  // whole workgroup
  const int N = f.N, C = f.C, NP = pad_tokens(N);
  const long long base = f.offset[t];
  const int nt = min(max(f.offset[t + 1] - int(base), 0), N);
  const long long total = min((long long)f.offset[f.T], f.B);
  // the rows the call may write (those past total were not formed either)
  const int nrow = int(max(0LL, min((long long)nt, total - base)));
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int c_lo = sl * rc_slice_width(C, S) + wave * kRcWaveCh;
  if (nrow == 0) return;  // whole workgroup
  // waves without channels stage operator entries and keep the barriers only
  const bool live = !(wave * kRcWaveCh >= rc_slice_width(C, S) || c_lo >= C);
  const int tid = threadIdx.x;
  const int r16 = lane & 15, g = lane >> 4;
  const int cw = c_lo + 8 * r16;  // the lane's first channel
  const int rb = C * 2;
  const __amdgpu_buffer_rsrc_t xres =
      make_rsrc(static_cast<const uint16_t*>(f.X) + size_t(t) * N * C, uint32_t(N) * rb);
  const __amdgpu_buffer_rsrc_t lres = make_rsrc(f.rows + size_t(base) * 2 * NP, uint32_t(nrow) * 4 * NP);
  const int vx = 8 * g * rb + (live && cw < C ? cw * 2 : kOOB);
  // staged operator entries: per buffer RT tiles x 2 parts x 16 rows of kBlk
  // tokens, each row kRowB bytes (16 more than its entries, so that the 16
  // rows read at once fall in distinct banks)
  constexpr int kBlk = 128;
  constexpr int kRowB = kBlk * 2 + 16;
  __shared__ __align__(16) char s_a[2][RT * 2 * 16 * kRowB];
  auto sweep = [&](auto tiles, int c0) __attribute__((always_inline)) {
    constexpr int NT = decltype(tiles)::value;
    constexpr int UPT = NT * 2 * 16 * 16 / (kRcWaves * kWave);  // 16-byte units a thread stages per block
    static_assert(UPT * kRcWaves * kWave == NT * 2 * 16 * 16, "whole units per thread");
    f32x4 acc[NT][8];
#pragma unroll
    for (int i = 0; i < NT; ++i)
#pragma unroll
      for (int c = 0; c < 8; ++c) acc[i][c] = f32x4{0.f, 0.f, 0.f, 0.f};
    auto loadx = [&](int k0, u32x4 (&x)[8]) __attribute__((always_inline)) {
#pragma unroll
      for (int e = 0; e < 8; ++e)
        x[e] = __builtin_amdgcn_raw_buffer_load_b128(xres, vx + __builtin_amdgcn_readfirstlane((k0 + e) * rb), 0, 0);
    };
    // unit q of a block: token group q % 16, row (q / 16) % 16, part (q / 256) % 2, tile q / 512
    // half hf of a block's units (UPT / 2 a thread)
    auto stage_load = [&](int blk, int hf, u32x4 (&u)[UPT / 2]) __attribute__((always_inline)) {
#pragma unroll
      for (int k2 = 0; k2 < UPT / 2; ++k2) {
        const int k = hf * (UPT / 2) + k2;
        const int q = tid + k * kRcWaves * kWave;
        const int uu = q & 15, r = (q >> 4) & 15, p = (q >> 8) & 1, i = q >> 9;
        const int tok = blk * kBlk + 8 * uu;
        const int off = (c0 + 16 * i + r) * 4 * NP + p * 2 * NP + 2 * tok;
        u[k2] = __builtin_amdgcn_raw_buffer_load_b128(lres, tok < NP ? off : kOOB, 0, 0);
      }
    };
    auto stage_store = [&](int buf, int hf, const u32x4 (&u)[UPT / 2]) __attribute__((always_inline)) {
#pragma unroll
      for (int k2 = 0; k2 < UPT / 2; ++k2) {
        const int k = hf * (UPT / 2) + k2;
        const int q = tid + k * kRcWaves * kWave;
        const int uu = q & 15, r = (q >> 4) & 15, p = (q >> 8) & 1, i = q >> 9;
        *reinterpret_cast<u32x4*>(&s_a[buf][((i * 2 + p) * 16 + r) * kRowB + uu * 16]) = u[k2];
      }
    };
    // one 32-token step at token kk of buffer buf's block
    auto step = [&](const u32x4 (&x)[8], int buf, int kk) __attribute__((always_inline)) {
      u32x4 ah[NT], al[NT];
#pragma unroll
      for (int i = 0; i < NT; ++i) {
        ah[i] = *reinterpret_cast<const u32x4*>(&s_a[buf][((i * 2 + 0) * 16 + r16) * kRowB + (kk + 8 * g) * 2]);
        al[i] = *reinterpret_cast<const u32x4*>(&s_a[buf][((i * 2 + 1) * 16 + r16) * kRowB + (kk + 8 * g) * 2]);
      }
#pragma unroll
      for (int c = 0; c < 8; ++c) {
        u32x4 wc;
#pragma unroll
        for (int j = 0; j < 4; ++j)
          wc[j] = __builtin_amdgcn_perm(x[2 * j + 1][c >> 1], x[2 * j][c >> 1], (c & 1) ? 0x07060302u : 0x05040100u);
        const bf16x8 bw = __builtin_bit_cast(bf16x8, wc);
#pragma unroll
        for (int i = 0; i < NT; ++i)
          acc[i][c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, ah[i]), bw, acc[i][c], 0, 0, 0);
#pragma unroll
        for (int i = 0; i < NT; ++i)
          acc[i][c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, al[i]), bw, acc[i][c], 0, 0, 0);
      }
    };
    const int nblk = (NP + kBlk - 1) / kBlk;
    u32x4 xa[8], xb[8], su[UPT / 2];
    if (live) {
      loadx(0, xa);
      __builtin_amdgcn_sched_barrier(0);
      loadx(32, xb);
    }
#pragma unroll
    for (int hf = 0; hf < 2; ++hf) {
      stage_load(0, hf, su);
      stage_store(0, hf, su);
    }
    lds_barrier();
    // block blk from buffer blk % 2 while the next block is staged into the
    // other, half of it in each half of the block's steps; one barrier a block
    for (int blk = 0; blk < nblk; ++blk) {
      const int buf = blk & 1;
      const bool next = blk + 1 < nblk;
#pragma unroll
      for (int hf = 0; hf < 2; ++hf) {
        if (next) stage_load(blk + 1, hf, su);
        const int k0 = blk * kBlk + 64 * hf;
        if (live && k0 < NP) {
          __builtin_amdgcn_sched_barrier(0);
          step(xa, buf, 64 * hf);
          loadx(k0 + 64, xa);
          __builtin_amdgcn_sched_barrier(0);
          if (k0 + 32 < NP) step(xb, buf, 64 * hf + 32);
          loadx(k0 + 96, xb);
        }
        if (next) stage_store(buf ^ 1, hf, su);
      }
      lds_barrier();
    }
    if (!live) return;
#pragma unroll
    for (int i = 0; i < NT; ++i) {
      // one descriptor per 16-row tile (the lanes' rows differ); its size
      // stops at the last row the call may write
      const long long row0 = base + c0 + 16 * i;
      const int rows = min(16, nrow - c0 - 16 * i);
      if (rows <= 0) break;
      const __amdgpu_buffer_rsrc_t ores =
          make_rsrc_uniform(static_cast<Out*>(f.out_tokens) + size_t(row0) * C, uint32_t(rows * C * sizeof(Out)));
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int rt = 4 * g + e;
        if (rt < rows) {
          float y8[8];
#pragma unroll
          for (int c = 0; c < 8; ++c) y8[c] = acc[i][c][e];
          if (cw < C) store8<Out>(ores, (rt * C + cw) * int(sizeof(Out)), y8);
        }
      }
    }
  };
  for (int c0 = 0; c0 < nrow; c0 += 16 * RT) {
    const int rtiles = (nrow - c0 + 15) / 16;  // uniform
    if (rtiles >= 3) sweep(std::integral_constant<int, 3>{}, c0);
    else if (rtiles == 2) sweep(std::integral_constant<int, 2>{}, c0);
    else sweep(std::integral_constant<int, 1>{}, c0);
  }
}

// dynamic LDS a workgroup may take (the static arrays use about 2 KB)
constexpr size_t kFilterLdsMax = (160 - 4) * 1024;

// rows per chunk: the most (32, 16 or 8) whose LDS fits
int filter_rows(int H, int W, int F, bool mfma, int det_levels = 0) {
  for (int kr = 32; kr >= 8; kr /= 2)
    if (filter_lds(H, W, F, kr, mfma, det_levels).bytes <= kFilterLdsMax) return kr;
  return 0;
}

// the row kernel: one workgroup per frame
void launch_filter_rows(const wz_config& c, const VideoArgs<FilterArgs>& va, int V, const Bank& bank, int det_levels,
                        hipStream_t s) {
  const dim3 grid(unsigned((c.T + kXcds - 1) / kXcds * kXcds), V), block(kFThreads);
  const int kr = filter_rows(c.H, c.W, bank.F, true, det_levels);
  const size_t lds = filter_lds(c.H, c.W, bank.F, kr, true, det_levels).bytes;
  if (kr == 32) hipLaunchKernelGGL((k_filter_assign<uint16_t, uint16_t, 32, true>), grid, block, lds, s, va, bank);
  else if (kr == 16) hipLaunchKernelGGL((k_filter_assign<uint16_t, uint16_t, 16, true>), grid, block, lds, s, va, bank);
  else hipLaunchKernelGGL((k_filter_assign<uint16_t, uint16_t, 8, true>), grid, block, lds, s, va, bank);
}

template <typename Out>
void launch_contract_typed(const wz_config& c, const VideoArgs<RowsArgs>& va, int V, hipStream_t s) {
  const int S = rc_slices(c.C);
  const dim3 grid(unsigned((c.T + kXcds - 1) / kXcds * kXcds * S), V), block(kRcWaves * kWave);
  hipLaunchKernelGGL((k_filter_contract<Out, 3>), grid, block, 0, s, va);
}

template <typename In, typename Out>
void launch_filter_typed(const wz_config& c, const VideoArgs<FilterArgs>& va, int V, const Bank& bank,
                         int det_levels, hipStream_t s) {
  constexpr bool mfma = sizeof(In) == 2;
  const int S = (c.C + filter_slice(mfma) - 1) / filter_slice(mfma);
  const dim3 grid(unsigned((c.T + kXcds - 1) / kXcds * kXcds * S), V), block(kFThreads);
  const int kr = filter_rows(c.H, c.W, bank.F, mfma, det_levels);
  const size_t lds = filter_lds(c.H, c.W, bank.F, kr, mfma, det_levels).bytes;
  if (kr == 32) hipLaunchKernelGGL((k_filter_assign<In, Out, 32>), grid, block, lds, s, va, bank);
  else if (kr == 16) hipLaunchKernelGGL((k_filter_assign<In, Out, 16>), grid, block, lds, s, va, bank);
  else hipLaunchKernelGGL((k_filter_assign<In, Out, 8>), grid, block, lds, s, va, bank);
}

}  // namespace

bool filter_assign_supported(const wz_config& c) {
  return c.H <= 64 && c.W <= 64 && c.H * c.W <= 1024 && filter_rows(c.H, c.W, kMaxTaps, true) > 0 &&
         filter_rows(c.H, c.W, kMaxTaps, false) > 0;
}

// The split form pays a second launch and a round trip of the rows through
// memory; it wins where the fused kernel's LDS holds full-frame rows for at
// most 16 kept tokens at a time (large frames), so that frames with more
// kept tokens would read their slice of X from memory once per chunk.
bool filter_split(const wz_config& c) {
  return c.spatial_basis != WZ_HAAR && c.in_dtype == WZ_BF16 && filter_rows(c.H, c.W, kMaxTaps, true) < 32;
}

bool filter_budget_folds(const wz_config& c) {
  if (c.T > kWave || c.temporal_basis != WZ_HAAR || c.spatial_basis == WZ_HAAR || !filter_assign_supported(c))
    return false;
  // only where the budget's LDS leaves the rows per chunk as they are
  const int F = make_bank(c.spatial_basis).F;
  const bool mf = c.in_dtype == WZ_BF16;
  return filter_rows(c.H, c.W, F, mf, c.levels) == filter_rows(c.H, c.W, F, mf) &&
         filter_rows(c.H, c.W, F, true, c.levels) == filter_rows(c.H, c.W, F, true);
}

size_t filter_rows_bytes(const wz_config& c) {
  return filter_split(c) ? size_t(c.B) * 4 * pad_tokens(c.H * c.W) : 0;
}

hipError_t launch_filter_assign(const wz_config& c, const void* X, const float* tok_score, const int32_t* offset,
                                const int32_t* rank, uint16_t* rows, void* out_tokens, int32_t* out_index,
                                hipStream_t s, const Videos& vs, const FoldedBudget& fb) {
  if (!filter_assign_supported(c) || c.spatial_basis == WZ_HAAR) return hipErrorInvalidValue;
  if (rows && c.in_dtype != WZ_BF16) return hipErrorInvalidValue;
  // budgets computed in the kernel: one wave, Haar temporal basis, with the
  // per-frame kernel's ranks; otherwise the offsets are given
  const bool wb = fb.rel != nullptr;
  if (wb ? (!filter_budget_folds(c) || !rank || !fb.delta || !fb.offset) : !offset) return hipErrorInvalidValue;
  const int det_levels = wb ? c.levels : 0;
  const Bank bank = make_bank(c.spatial_basis);
  VideoArgs<FilterArgs> va{};
  for (int v = 0; v < vs.V; ++v) {
    FilterArgs& a = va.v[v];
    a.X = advance(X, v * vs.x);
    a.tok_score = advance(tok_score, v * vs.ws);
    a.offset = wb ? nullptr : advance(offset, v * vs.off);
    a.rel = wb ? advance(fb.rel, v * vs.ws) : nullptr;
    a.delta = wb ? advance(fb.delta, v * vs.ws) : nullptr;
    a.budget_out = wb ? advance(fb.budget, v * vs.bud) : nullptr;
    a.offset_out = wb ? advance(fb.offset, v * vs.off) : nullptr;
    a.rank = advance(rank, v * vs.ws);
    a.rows = advance(rows, v * vs.ws);
    a.out_tokens = advance(out_tokens, v * vs.out);
    a.out_index = advance(out_index, v * vs.idx);
    a.B = c.B;
    a.T = c.T;
    a.H = c.H;
    a.W = c.W;
    a.C = c.C;
    a.levels = c.levels;
    a.lam = c.lambda_;
    a.tau = c.tau;
  }
  if (rows) {
    // split form: the rows once per frame, then the contraction per slice
    launch_filter_rows(c, va, vs.V, bank, det_levels, s);
    VideoArgs<RowsArgs> ra{};
    for (int v = 0; v < vs.V; ++v) {
      RowsArgs& a = ra.v[v];
      a.X = va.v[v].X;
      a.offset = wb ? va.v[v].offset_out : va.v[v].offset;
      a.rows = va.v[v].rows;
      a.out_tokens = va.v[v].out_tokens;
      a.B = c.B;
      a.T = c.T;
      a.N = c.H * c.W;
      a.C = c.C;
    }
    if (c.out_dtype == WZ_BF16) launch_contract_typed<uint16_t>(c, ra, vs.V, s);
    else launch_contract_typed<float>(c, ra, vs.V, s);
  } else if (c.in_dtype == WZ_BF16) {
    if (c.out_dtype == WZ_BF16) launch_filter_typed<uint16_t, uint16_t>(c, va, vs.V, bank, det_levels, s);
    else launch_filter_typed<uint16_t, float>(c, va, vs.V, bank, det_levels, s);
  } else {
    if (c.out_dtype == WZ_BF16) launch_filter_typed<float, uint16_t>(c, va, vs.V, bank, det_levels, s);
    else launch_filter_typed<float, float>(c, va, vs.V, bank, det_levels, s);
  }
  return hipGetLastError();
}

}  // namespace wz
