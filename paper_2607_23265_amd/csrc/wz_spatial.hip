// Stage 3: Wavelet Spatial Modulator (Eq. (7), Eq. (12)-(15)) and the Token
// Assigner's compaction (Eq. (19)), with the interpolation of Eq. (17)
// replaced by saliency-ranked selection.
//
// Grid: `sub` workgroups of 4 waves per frame.  Each workgroup of frame t
//   1. loads the frame's scores a_{t,.} into LDS and forms the saliency map
//      M = min-max(a) (Eq. (7); M = 0 if all scores are equal);
//   2. marks the budget[t] highest-scoring tokens (ties: smaller index) and
//      lists them in raster order (block prefix scan);
//   3. gives each wave one kept token at a time: it reads the token's 2x2 Haar block (the last
//      row / column repeated when H or W is odd), forms LL, LH, HL, HH with the
//      orthonormal 2-D Haar butterflies (Eq. (12)), multiplies LH, HL, HH by
//      g = lambda * mean(M over the block) (Eq. (13)-(14)), inverts for the
//      token's position in the block (Eq. (15)) and writes the row to
//      out_tokens[offset[t] + k] and its flat index to out_index.
// Only the blocks of kept tokens are touched: the second read of X is at most
// 4 * B tokens, and usually hits the Infinity Cache right after stage 1.
#include <algorithm>

#include "wz_internal.h"

namespace wz {
namespace {

constexpr int kThreads = 256;
constexpr int kNMax = 4096;

template <typename In>
struct Load8;
template <>
struct Load8<uint16_t> {  // 8 bf16 channels = 16 bytes
  static constexpr int kV = 8;
  __device__ static void run(const uint16_t* p, float* v) {
    const u32x4 x = *reinterpret_cast<const u32x4*>(p);
#pragma unroll
    for (int i = 0; i < 4; ++i) { v[2 * i] = bf16_lo(x[i]); v[2 * i + 1] = bf16_hi(x[i]); }
  }
};
template <>
struct Load8<float> {  // 4 fp32 channels = 16 bytes
  static constexpr int kV = 4;
  __device__ static void run(const float* p, float* v) {
    const f32x4 x = *reinterpret_cast<const f32x4*>(p);
    v[0] = x[0]; v[1] = x[1]; v[2] = x[2]; v[3] = x[3];
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
  typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
  u32x2 o;
  o[0] = f32_to_bf16_rne(v[0]) | (f32_to_bf16_rne(v[1]) << 16);
  o[1] = f32_to_bf16_rne(v[2]) | (f32_to_bf16_rne(v[3]) << 16);
  *reinterpret_cast<u32x2*>(p) = o;
}

__device__ __forceinline__ int block_scan_excl(int v, int& total, int* red) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int inc = v;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const int o = __shfl_up(inc, d, kWave);
    if (lane >= d) inc += o;
  }
  __syncthreads();
  if (lane == 63) red[wave] = inc;
  __syncthreads();
  int before = 0;
  total = 0;
#pragma unroll
  for (int i = 0; i < kThreads / kWave; ++i) {
    if (i < wave) before += red[i];
    total += red[i];
  }
  return before + inc - v;
}

template <typename In, typename Out>
__global__ __launch_bounds__(kThreads) void k_spatial_condense(const In* __restrict__ X,
                                                               const float* __restrict__ tok_score,
                                                               const int32_t* __restrict__ budget,
                                                               const int32_t* __restrict__ offset, int H,
                                                               int W, int C, long long B, float lam, int sub,
                                                               Out* __restrict__ out_tokens,
                                                               int32_t* __restrict__ out_index) {
  constexpr int V = Load8<In>::kV;
  __shared__ float s_m[kNMax];
  __shared__ unsigned char s_flag[kNMax];
  __shared__ int s_kept[kNMax];
  __shared__ float s_red[2][kThreads / kWave];
  __shared__ int s_ired[kThreads / kWave];

  const int t = blockIdx.x / sub;
  const int part = blockIdx.x % sub;
  const int N = H * W;
  const int nt = min(budget[t], N);
  const int base = offset[t];
  if (nt <= 0 || base < 0 || base >= B) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const float* a = tok_score + size_t(t) * N;

  float lo = INFINITY, hi = -INFINITY;
  for (int n = tid; n < N; n += kThreads) {
    const float v = a[n];
    s_m[n] = v;
    lo = fminf(lo, v);
    hi = fmaxf(hi, v);
  }
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) {
    lo = fminf(lo, __shfl_xor(lo, m, kWave));
    hi = fmaxf(hi, __shfl_xor(hi, m, kWave));
  }
  if (lane == 0) { s_red[0][wave] = lo; s_red[1][wave] = hi; }
  __syncthreads();
  lo = s_red[0][0];
  hi = s_red[1][0];
#pragma unroll
  for (int i = 1; i < kThreads / kWave; ++i) { lo = fminf(lo, s_red[0][i]); hi = fmaxf(hi, s_red[1][i]); }

  // Selection: token n is kept iff fewer than nt tokens beat it, where k beats n
  // when a_k > a_n or (a_k == a_n and k < n).
  for (int n = tid; n < N; n += kThreads) {
    unsigned char keep = 1;
    if (nt < N) {
      const float an = s_m[n];
      int rank = 0;
      for (int j = 0; j < N; ++j) {
        const float aj = s_m[j];
        rank += (aj > an) || (aj == an && j < n);
      }
      keep = rank < nt;
    }
    s_flag[n] = keep;
  }
  __syncthreads();
  // list the kept tokens in raster order: thread tid scans a contiguous chunk
  const int chunk = (N + kThreads - 1) / kThreads;
  const int n0 = min(N, tid * chunk), n1 = min(N, n0 + chunk);
  int cnt = 0;
  for (int n = n0; n < n1; ++n) cnt += s_flag[n];
  int total = 0;
  int pos = block_scan_excl(cnt, total, s_ired);
  for (int n = n0; n < n1; ++n)
    if (s_flag[n]) s_kept[pos++] = n;
  // saliency map M (Eq. (7)); every thread has finished ranking (barrier in the scan)
  const float range = hi - lo;
  for (int n = tid; n < N; n += kThreads) s_m[n] = range > 0.f ? (s_m[n] - lo) / range : 0.f;
  __syncthreads();

  const In* Xt = X + size_t(t) * N * C;
  const int nvec = C / V;
  // rows beyond the kept count or beyond B are never written
  const int rows = int(min((long long)min(nt, total), B - base));
  constexpr int kWaves = kThreads / kWave;
  constexpr int UNR = 4;  // channel vectors per lane in flight (4 loads each)
  for (int k = part * kWaves + wave; k < rows; k += sub * kWaves) {
    const int n = s_kept[k];
    const int h = n / W, w = n - h * W;
    const int i0 = h & ~1, j0 = w & ~1;
    const int i1 = min(i0 + 1, H - 1), j1 = min(j0 + 1, W - 1);
    const float g = lam * (0.25f * (((s_m[i0 * W + j0] + s_m[i0 * W + j1]) + s_m[i1 * W + j0]) + s_m[i1 * W + j1]));
    const float sw = (w & 1) ? -1.f : 1.f;
    const float sh = (h & 1) ? -1.f : 1.f;
    const In* p00 = Xt + size_t(i0 * W + j0) * C;
    const In* p01 = Xt + size_t(i0 * W + j1) * C;
    const In* p10 = Xt + size_t(i1 * W + j0) * C;
    const In* p11 = Xt + size_t(i1 * W + j1) * C;
    Out* dst = out_tokens + size_t(base + k) * C;
    for (int v0 = lane; v0 < nvec; v0 += UNR * kWave) {
      float x00[UNR][V], x01[UNR][V], x10[UNR][V], x11[UNR][V];
#pragma unroll
      for (int u = 0; u < UNR; ++u) {
        const int v = v0 + u * kWave;
        if (v < nvec) {
          Load8<In>::run(p00 + v * V, x00[u]);
          Load8<In>::run(p01 + v * V, x01[u]);
          Load8<In>::run(p10 + v * V, x10[u]);
          Load8<In>::run(p11 + v * V, x11[u]);
        }
      }
#pragma unroll
      for (int u = 0; u < UNR; ++u) {
        const int v = v0 + u * kWave;
        if (v >= nvec) break;
        float y[V];
#pragma unroll
        for (int i = 0; i < V; ++i) {
          // orthonormal 2-D Haar butterflies of the block (Eq. (12))
          const float LL = 0.5f * ((x00[u][i] + x01[u][i]) + (x10[u][i] + x11[u][i]));
          const float LH = 0.5f * ((x00[u][i] - x01[u][i]) + (x10[u][i] - x11[u][i]));
          const float HL = 0.5f * ((x00[u][i] + x01[u][i]) - (x10[u][i] + x11[u][i]));
          const float HH = 0.5f * ((x00[u][i] - x01[u][i]) - (x10[u][i] - x11[u][i]));
          // gate the detail bands (Eq. (14)) and invert at the token's position (Eq. (15))
          y[i] = 0.5f * (LL + g * (sw * LH + sh * HL + (sw * sh) * HH));
        }
        store_row<Out, V>(dst + v * V, y);
      }
    }
    if (lane == 0) out_index[base + k] = t * N + n;
  }
}

template <typename In, typename Out>
void launch_typed(const wz_config& c, const void* X, const float* tok_score, const int32_t* budget,
                  const int32_t* offset, void* out_tokens, int32_t* out_index, hipStream_t s) {
  // one wave per kept row: about B / T rows per frame, 4 waves per workgroup
  const long long per_frame = (c.B + c.T - 1) / c.T;
  const int sub = int(std::max<long long>(1, std::min<long long>(64, (per_frame + 3) / 4)));
  hipLaunchKernelGGL((k_spatial_condense<In, Out>), dim3(c.T * sub), dim3(kThreads), 0, s,
                     static_cast<const In*>(X), tok_score, budget, offset, c.H, c.W, c.C, (long long)c.B, c.lambda_, sub,
                     static_cast<Out*>(out_tokens), out_index);
}

}  // namespace

hipError_t launch_spatial_condense(const wz_config& c, const void* X, const float* tok_score,
                                   const int32_t* budget, const int32_t* offset, void* out_tokens,
                                   int32_t* out_index, hipStream_t s) {
  if (c.in_dtype == WZ_BF16) {
    if (c.out_dtype == WZ_BF16) launch_typed<uint16_t, uint16_t>(c, X, tok_score, budget, offset, out_tokens, out_index, s);
    else launch_typed<uint16_t, float>(c, X, tok_score, budget, offset, out_tokens, out_index, s);
  } else {
    if (c.out_dtype == WZ_BF16) launch_typed<float, uint16_t>(c, X, tok_score, budget, offset, out_tokens, out_index, s);
    else launch_typed<float, float>(c, X, tok_score, budget, offset, out_tokens, out_index, s);
  }
  return hipGetLastError();
}

}  // namespace wz
