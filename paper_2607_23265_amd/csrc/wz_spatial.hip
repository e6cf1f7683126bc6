// Stage 3: Wavelet Spatial Modulator (Eq. (12)-(15)) and the Token Assigner's
// compaction (Eq. (19)), with the interpolation of Eq. (17) replaced by
// saliency-ranked selection.
//
// One wave per output row k < offset[T], every wave on its own (no LDS, no
// barrier):
//   1. its frame t is the number of frames whose offset is <= k, minus one
//      (one ballot per 64 frames); the frame keeps n_t = offset[t+1] -
//      offset[t] tokens and row k is its (k - offset[t])-th in raster order;
//   2. the kept tokens are those of selection rank < n_t (ranks and the
//      saliency map M_t come from the frame preparation); ballots over the
//      ranks, 64 tokens at a time, find the row's token n;
//   3. it reads the token's 2x2 Haar block (the last row / column repeated
//      when H or W is odd) and M over the block, forms LL, LH, HL, HH with the
//      orthonormal 2-D Haar butterflies (Eq. (12)), multiplies LH, HL, HH by
//      g = lambda * mean(M over the block) (Eq. (13)-(14)), inverts for the
//      token's position in the block (Eq. (15)) and writes the row to
//      out_tokens[k] and t*H*W + n to out_index[k].
// Only the blocks of kept tokens are touched: the second read of X is at most
// 4 * B tokens, and usually hits the Infinity Cache right after stage 1.
#include <algorithm>

#include "wz_device.h"

namespace wz {
namespace {

constexpr int kThreads = 256;

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

// FC: 64-frame chunks of offset[] read per wave (T <= 64 * FC); UNR:
// 16-byte channel vectors per lane and input row in flight (the four rows of
// the block are read at once).
template <typename In, typename Out, int UNR, int FC>
__global__ __launch_bounds__(kThreads) void k_spatial_gather(const In* __restrict__ X,
                                                             const int32_t* __restrict__ rank,
                                                             const float* __restrict__ sal,
                                                             const int32_t* __restrict__ offset, int T, int H,
                                                             int W, int C, long long B, float lam,
                                                             Out* __restrict__ out_tokens,
                                                             int32_t* __restrict__ out_index) {
  constexpr int V = Vec16<In>::kV;
  constexpr int kWaves = kThreads / kWave;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const long long k = (long long)blockIdx.x * kWaves + wave;  // output row
  const int N = H * W;

  // 1. frame of row k (offset is nondecreasing from offset[0] = 0)
  const __amdgpu_buffer_rsrc_t ores = make_rsrc(offset, uint32_t(T + 1) * 4);
  int ov[FC];
#pragma unroll
  for (int c = 0; c < FC; ++c) {
    const int i = c * kWave + lane;
    ov[c] = int(__builtin_amdgcn_raw_buffer_load_b32(ores, i < T ? i * 4 : kOOB, 0, 0));
  }
  const long long total = min((long long)offset[T], B);
  if (k >= total) return;
  int cnt = 0;
#pragma unroll
  for (int c = 0; c < FC; ++c) cnt += __popcll(__ballot(c * kWave + lane < T && ov[c] <= k));
  const int t = cnt - 1;
  if (t < 0) return;
  const int base = offset[t];
  const int nt = min(offset[t + 1] - base, N);
  const int p = int(k - base);
  if (p >= nt) return;

  // 2. the p-th kept token of frame t in raster order
  const __amdgpu_buffer_rsrc_t rres = make_rsrc(rank + size_t(t) * N, uint32_t(N) * 4);
  int n = -1, before = 0;
  for (int c0 = 0; c0 < N && n < 0; c0 += 8 * kWave) {
    int rv[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int i = c0 + u * kWave + lane;
      rv[u] = int(__builtin_amdgcn_raw_buffer_load_b32(rres, i < N ? i * 4 : kOOB, 0, 0));
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int i = c0 + u * kWave + lane;
      const bool kept = i < N && rv[u] < nt;
      const uint64_t m = __ballot(kept);
      const int pc = __popcll(m);
      if (n < 0 && p < before + pc) {
        const int j = p - before;  // the j-th set bit of m
        const uint64_t below = lane ? (m << (64 - lane)) : 0ull;  // bits of the lanes under this one
        const uint64_t sel = __ballot(kept && __popcll(below) == j);
        n = c0 + u * kWave + __builtin_ctzll(sel);
      }
      before += pc;
    }
  }
  if (n < 0) return;

  // 3. the block, its saliency gate and the reconstruction
  const int h = n / W, w = n - h * W;
  const int i0 = h & ~1, j0 = w & ~1;
  const int i1 = min(i0 + 1, H - 1), j1 = min(j0 + 1, W - 1);
  const float* st = sal + size_t(t) * N;
  const float m00 = st[i0 * W + j0], m01 = st[i0 * W + j1], m10 = st[i1 * W + j0], m11 = st[i1 * W + j1];
  const __amdgpu_buffer_rsrc_t xres = make_rsrc(X + size_t(t) * N * C, uint32_t(N) * C * sizeof(In));
  const int r00 = (i0 * W + j0) * C * int(sizeof(In)), r01 = (i0 * W + j1) * C * int(sizeof(In));
  const int r10 = (i1 * W + j0) * C * int(sizeof(In)), r11 = (i1 * W + j1) * C * int(sizeof(In));
  const float sw = (w & 1) ? -1.f : 1.f;
  const float sh = (h & 1) ? -1.f : 1.f;
  Out* dst = out_tokens + size_t(k) * C;
  const int nvec = C / V;
  for (int v0 = lane; v0 < nvec; v0 += UNR * kWave) {
    u32x4 x[UNR][4];
#pragma unroll
    for (int u = 0; u < UNR; ++u) {
      const int v = v0 + u * kWave;
      const int cb = v < nvec ? v * 16 : kOOB;
      x[u][0] = __builtin_amdgcn_raw_buffer_load_b128(xres, r00 + cb, 0, 0);
      x[u][1] = __builtin_amdgcn_raw_buffer_load_b128(xres, r01 + cb, 0, 0);
      x[u][2] = __builtin_amdgcn_raw_buffer_load_b128(xres, r10 + cb, 0, 0);
      x[u][3] = __builtin_amdgcn_raw_buffer_load_b128(xres, r11 + cb, 0, 0);
    }
    const float g = lam * (0.25f * (((m00 + m01) + m10) + m11));
#pragma unroll
    for (int u = 0; u < UNR; ++u) {
      const int v = v0 + u * kWave;
      float x00[V], x01[V], x10[V], x11[V], y[V];
      Vec16<In>::widen(x[u][0], x00);
      Vec16<In>::widen(x[u][1], x01);
      Vec16<In>::widen(x[u][2], x10);
      Vec16<In>::widen(x[u][3], x11);
#pragma unroll
      for (int i = 0; i < V; ++i) {
        // orthonormal 2-D Haar butterflies of the block (Eq. (12))
        const float LL = 0.5f * ((x00[i] + x01[i]) + (x10[i] + x11[i]));
        const float LH = 0.5f * ((x00[i] - x01[i]) + (x10[i] - x11[i]));
        const float HL = 0.5f * ((x00[i] + x01[i]) - (x10[i] + x11[i]));
        const float HH = 0.5f * ((x00[i] - x01[i]) - (x10[i] - x11[i]));
        // gate the detail bands (Eq. (14)) and invert at the token's position (Eq. (15))
        y[i] = 0.5f * (LL + g * (sw * LH + sh * HL + (sw * sh) * HH));
      }
      if (v < nvec) store_row<Out, V>(dst + v * V, y);
    }
  }
  if (lane == 0) out_index[k] = t * N + n;
}

template <typename In, typename Out, int FC>
void launch_typed(const wz_config& c, const void* X, const int32_t* rank, const float* sal, const int32_t* offset,
                  void* out_tokens, int32_t* out_index, hipStream_t s) {
  const int nvec = c.C / Vec16<In>::kV;
  const int vec_per_lane = (nvec + kWave - 1) / kWave;
  const long long rows = c.B;
  const dim3 grid(unsigned((rows + kThreads / kWave - 1) / (kThreads / kWave))), block(kThreads);
  const In* x = static_cast<const In*>(X);
  Out* o = static_cast<Out*>(out_tokens);
#define WZ_GATHER(U)                                                                                       \
  hipLaunchKernelGGL((k_spatial_gather<In, Out, U, FC>), grid, block, 0, s, x, rank, sal, offset, c.T, c.H, \
                     c.W, c.C, (long long)c.B, c.lambda_, o, out_index)
  // at most 4 vectors per lane and row in flight: deeper batches of every
  // wave's four rows overfill the CU's L1 with misses and run slower
  if (vec_per_lane <= 1) WZ_GATHER(1);
  else if (vec_per_lane <= 2) WZ_GATHER(2);
  else WZ_GATHER(4);
#undef WZ_GATHER
}

template <typename In, typename Out>
void launch_frames(const wz_config& c, const void* X, const int32_t* rank, const float* sal, const int32_t* offset,
                   void* out_tokens, int32_t* out_index, hipStream_t s) {
  if (c.T <= 64) launch_typed<In, Out, 1>(c, X, rank, sal, offset, out_tokens, out_index, s);
  else if (c.T <= 256) launch_typed<In, Out, 4>(c, X, rank, sal, offset, out_tokens, out_index, s);
  else launch_typed<In, Out, kMaxFrames / kWave>(c, X, rank, sal, offset, out_tokens, out_index, s);
}

}  // namespace

hipError_t launch_spatial_gather(const wz_config& c, const void* X, const int32_t* rank, const float* sal,
                                 const int32_t* offset, void* out_tokens, int32_t* out_index, hipStream_t s) {
  if (c.B == 0) return hipGetLastError();
  if (c.in_dtype == WZ_BF16) {
    if (c.out_dtype == WZ_BF16) launch_frames<uint16_t, uint16_t>(c, X, rank, sal, offset, out_tokens, out_index, s);
    else launch_frames<uint16_t, float>(c, X, rank, sal, offset, out_tokens, out_index, s);
  } else {
    if (c.out_dtype == WZ_BF16) launch_frames<float, uint16_t>(c, X, rank, sal, offset, out_tokens, out_index, s);
    else launch_frames<float, float>(c, X, rank, sal, offset, out_tokens, out_index, s);
  }
  return hipGetLastError();
}

}  // namespace wz
