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
// Workgroup (frame t, slice of 512 channels), 256 threads:
//   1. ranks the frame's tokens from their scores (wz_rank.h) and lists its
//      n_t kept tokens (rank < n_t) in raster order;
//   2. forms G and the per-axis analysis rows a_u in LDS;
//   3. per chunk of KR kept tokens builds their rows L_p in LDS (fp32,
//      through the partial sums B_i(w') = sum_j over the width), then each of
//      the 4 waves contracts KR / 4 of them with the frame's slice, one
//      16-byte vector of 8 channels per lane (fp32 accumulation), and writes
//      the rows to out_tokens[offset_t + k] (k = raster position among the
//      kept tokens), their flat indices to out_index.
// The frame's slice is read once per chunk of KR kept tokens (from L2 after
// the first).  Supported: H, W <= 64, H*W <= 1024 (the host checks).
#include "wz_rank.h"
#include "wz_wavelets.h"

namespace wz {
namespace {

constexpr int kFThreads = 256;
constexpr int kFWaves = kFThreads / kWave;
constexpr int kFSlice = kWave * 8;  // channels of a workgroup: 8 per lane
constexpr int kMaxAct = kMaxTaps / 2;  // synthesis rows touching one output sample

struct FilterArgs {
  const void* X;            // [T][H][W][C]
  const float* tok_score;   // [T][H*W]
  const int32_t* offset;    // [T+1]
  void* out_tokens;         // [B][C]
  int32_t* out_index;       // [B]
  long long B;
  int T, H, W, C;
  float lam;
};
static_assert(sizeof(VideoArgs<FilterArgs>) <= 4096, "per-video arguments exceed the kernel argument limit");

// 8 channels of a token row as floats.
template <typename In>
__device__ __forceinline__ void load8(__amdgpu_buffer_rsrc_t r, int off, float (&v)[8]);
template <>
__device__ __forceinline__ void load8<uint16_t>(__amdgpu_buffer_rsrc_t r, int off, float (&v)[8]) {
  const u32x4 x = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
#pragma unroll
  for (int i = 0; i < 4; ++i) { v[2 * i] = bf16_lo(x[i]); v[2 * i + 1] = bf16_hi(x[i]); }
}
template <>
__device__ __forceinline__ void load8<float>(__amdgpu_buffer_rsrc_t r, int off, float (&v)[8]) {
  const u32x4 x = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
  const u32x4 y = __builtin_amdgcn_raw_buffer_load_b128(r, off + 16, 0, 0);
#pragma unroll
  for (int i = 0; i < 4; ++i) { v[i] = __uint_as_float(x[i]); v[4 + i] = __uint_as_float(y[i]); }
}
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

// Bytes of dynamic LDS for a frame of H x W tokens and chunks of kr rows.
__host__ __device__ inline size_t filter_lds_bytes(int H, int W, int F, int kr) {
  const size_t N = size_t(H) * W, nh = bank_len(H, F), nw = bank_len(W, F);
  return N * 24                                   // ranking: key, rank, byrank, gate, order
         + N * 4 * 2                              // saliency, kept list
         + nh * nw * 4                            // gates
         + (2 * nh * H + 2 * nw * W) * 4          // analysis rows, both axes
         + size_t(kr) * 2 * kMaxAct * W * 4       // partial sums B1, B2
         + N * kr * 4;                            // operator rows
}

template <typename In, typename Out, int KR>
__global__ __launch_bounds__(kFThreads) void k_filter_assign(const VideoArgs<FilterArgs> va, const Bank bank) {
  constexpr int RW = KR / kFWaves;  // rows a wave contracts
  const FilterArgs& f = va.v[blockIdx.y];
  const int S = (f.C + kFSlice - 1) / kFSlice;
  const int b = blockIdx.x, xcd = b % kXcds, slot = b / kXcds;
  const int t = (slot / S) * kXcds + xcd, sl = slot % S;
  if (t >= f.T) return;  // whole workgroup
  const int H = f.H, W = f.W, N = H * W, F = bank.F, C = f.C;
  const int nh = bank_len(H, F), nw = bank_len(W, F);
  const long long base = f.offset[t];
  const int nt = min(max(f.offset[t + 1] - int(base), 0), N);
  const long long total = min((long long)f.offset[f.T], f.B);
  if (nt == 0) return;  // whole workgroup
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;

  extern __shared__ __align__(16) char s_dyn[];
  __shared__ int s_start[kBins], s_fill[kBins];
  __shared__ float s_mm[2 * kFWaves];
  __shared__ int s_wsum[kFWaves];
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
  float* s_M = reinterpret_cast<float*>(rl.order + N);  // [N] saliency M
  int32_t* s_kept = reinterpret_cast<int32_t*>(s_M + N);  // [nt] kept tokens in raster order
  float* s_G = reinterpret_cast<float*>(s_kept + N);    // [nh][nw] gates
  float* s_AH = s_G + nh * nw;                          // [2][nh][H] analysis rows along the height
  float* s_AW = s_AH + 2 * nh * H;                      // [2][nw][W] along the width
  float* s_B = s_AW + 2 * nw * W;                       // [KR][2][kMaxAct][W]
  float* s_L = s_B + KR * 2 * kMaxAct * W;              // [N][KR] operator rows, token-major

  // ---- 1. ranks from the scores; kept tokens in raster order ----
  {
    const __amdgpu_buffer_rsrc_t ares = make_rsrc(f.tok_score + size_t(t) * N, uint32_t(N) * 4);
    float lo = INFINITY, hi = -INFINITY;
    for (int n0 = 0; n0 < N; n0 += 4 * kFThreads) {
      float av[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int n = n0 + u * kFThreads + tid;
        av[u] = buf_load_f32(ares, n < N ? n * 4 : kOOB);
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int n = n0 + u * kFThreads + tid;
        if (n < N) {
          rl.key[n] = sel_key(av[u], n);
          lo = fminf(lo, av[u]);
          hi = fmaxf(hi, av[u]);
        }
      }
    }
    rank_frame<kFThreads>(N, H, W, f.lam, lo, hi, rl);
  }
  __syncthreads();
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
  __syncthreads();

  // synthesis weight of coefficient i (band u) at output position x of an
  // axis; 0 outside the filter
  auto syn = [&](int u, int x, int i) {
    const int k = x + F - 2 - 2 * i;
    return (k >= 0 && k < F) ? float(u == 0 ? bank.rec_lo[k] : bank.rec_hi[k]) : 0.f;
  };
  // first coefficient whose synthesis filter reaches position x (at most
  // kMaxAct of them, up to i0 + kMaxAct - 1)
  auto first_coef = [](int x) { return x >= 1 ? x / 2 : 0; };

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
        const int i = first_coef(h) + ii;
        if (i < nh) {
          const int j0 = first_coef(w);
          for (int jj = 0; jj < kMaxAct; ++jj) {
            const int j = j0 + jj;
            if (j >= nw) break;
            const float e = syn(0, w, j) * s_AW[j * W + x];
            const float pp = e + syn(1, w, j) * s_AW[(nw + j) * W + x];
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
    // ---- 3b. L_p(h', w') = sum_i E_i(h') B1_i(w') + P_i(h') B2_i(w') ----
    for (int q = tid; q < N * KR; q += kFThreads) {
      const int n = q / KR, r = q - n * KR, y = n / W, x = n - y * W;
      float s = 0.f;
      if (c0 + r < nt) {
        const int p = s_kept[c0 + r], h = p / W;
        const int i0 = first_coef(h);
        for (int ii = 0; ii < kMaxAct; ++ii) {
          const int i = i0 + ii;
          if (i >= nh) break;
          const float e = syn(0, h, i) * s_AH[i * H + y];
          const float pp = e + syn(1, h, i) * s_AH[(nh + i) * H + y];
          s += e * s_B[((r * 2 + 0) * kMaxAct + ii) * W + x] + pp * s_B[((r * 2 + 1) * kMaxAct + ii) * W + x];
        }
      }
      s_L[q] = s;
    }
    __syncthreads();
    // ---- 3c. the wave's RW rows against the frame's slice ----
    float acc[RW][8];
#pragma unroll
    for (int r = 0; r < RW; ++r)
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[r][e] = 0.f;
    constexpr int D = 4;  // tokens whose loads are in flight ahead
    float xv[D][8];
#pragma unroll
    for (int d = 0; d < D; ++d) load8<In>(xres, d < N ? d * rb + xoff : kOOB, xv[d]);
    for (int n0 = 0; n0 < N; n0 += D) {
#pragma unroll
      for (int d = 0; d < D; ++d) {
        const int n = n0 + d;
        float xc[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) xc[e] = xv[d][e];
        load8<In>(xres, n + D < N ? (n + D) * rb + xoff : kOOB, xv[d]);
        if (n < N) {
          const float* Lr = s_L + n * KR + wave * RW;
#pragma unroll
          for (int r = 0; r < RW; ++r) {
            const float l = Lr[r];
#pragma unroll
            for (int e = 0; e < 8; ++e) acc[r][e] = fmaf(l, xc[e], acc[r][e]);
          }
        }
      }
    }
#pragma unroll
    for (int r = 0; r < RW; ++r) {
      const int k = c0 + wave * RW + r;
      if (k < nt && base + k < total) {
        const __amdgpu_buffer_rsrc_t ores = make_rsrc_uniform(
            static_cast<Out*>(f.out_tokens) + size_t(base + k) * C, uint32_t(C) * sizeof(Out));
        if (vok) store8<Out>(ores, v * 8 * int(sizeof(Out)), acc[r]);
        if (sl == 0 && lane == 0) f.out_index[base + k] = t * N + s_kept[k];
      }
    }
    __syncthreads();  // the next chunk rewrites B and L
  }
}

template <typename In, typename Out>
void launch_filter_typed(const wz_config& c, const VideoArgs<FilterArgs>& va, int V, const Bank& bank,
                         hipStream_t s) {
  const int S = (c.C + kFSlice - 1) / kFSlice;
  const dim3 grid(unsigned((c.T + kXcds - 1) / kXcds * kXcds * S), V), block(kFThreads);
  if (c.H * c.W <= 512)
    hipLaunchKernelGGL((k_filter_assign<In, Out, 32>), grid, block, filter_lds_bytes(c.H, c.W, bank.F, 32), s, va,
                       bank);
  else
    hipLaunchKernelGGL((k_filter_assign<In, Out, 16>), grid, block, filter_lds_bytes(c.H, c.W, bank.F, 16), s, va,
                       bank);
}

}  // namespace

bool filter_assign_supported(const wz_config& c) {
  return c.H <= 64 && c.W <= 64 && c.H * c.W <= 1024;
}

hipError_t launch_filter_assign(const wz_config& c, const void* X, const float* tok_score, const int32_t* offset,
                                void* out_tokens, int32_t* out_index, hipStream_t s, const Videos& vs) {
  if (!filter_assign_supported(c) || c.spatial_basis == WZ_HAAR) return hipErrorInvalidValue;
  const Bank bank = make_bank(c.spatial_basis);
  VideoArgs<FilterArgs> va{};
  for (int v = 0; v < vs.V; ++v) {
    FilterArgs& a = va.v[v];
    a.X = advance(X, v * vs.x);
    a.tok_score = advance(tok_score, v * vs.ws);
    a.offset = advance(offset, v * vs.off);
    a.out_tokens = advance(out_tokens, v * vs.out);
    a.out_index = advance(out_index, v * vs.idx);
    a.B = c.B;
    a.T = c.T;
    a.H = c.H;
    a.W = c.W;
    a.C = c.C;
    a.lam = c.lambda_;
  }
  if (c.in_dtype == WZ_BF16) {
    if (c.out_dtype == WZ_BF16) launch_filter_typed<uint16_t, uint16_t>(c, va, vs.V, bank, s);
    else launch_filter_typed<uint16_t, float>(c, va, vs.V, bank, s);
  } else {
    if (c.out_dtype == WZ_BF16) launch_filter_typed<float, uint16_t>(c, va, vs.V, bank, s);
    else launch_filter_typed<float, float>(c, va, vs.V, bank, s);
  }
  return hipGetLastError();
}

}  // namespace wz
