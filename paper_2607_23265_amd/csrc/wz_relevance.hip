// Stage 1: similarity-branch Cross-Modal Scorer (Sec. 3.2.1) and Visual Change
// Estimator (Sec. 3.2.2, Eq. (8)) in ONE kernel that streams the frames once.
//
// Per token:  a_{t,n} = max_j (x . q_j) / (|x| |q_j|)
// Per frame:  p_t = sum_n x_{t,n} (the mean's cosine is the sum's),
//             r_t = max_j (p_t . q_j) / (|p_t| |q_j|),
//             delta_t = clamp(1 - cos(p_t, p_{t-1}), 0, 2), delta_0 = 0,
// with cos := 0 (so a = 0, r = 0, delta = 1) when a vector is zero.
//
// Work decomposition (MFMA path: bf16 inputs, Q >= 16, frames of >= 49 tokens).
// A workgroup owns a token tile of one frame (the whole frame when H*W <= 256;
// one wave per two 16-row MFMA tiles) and a slice of the channels.  The query is
// the operand every workgroup needs in full for its channels, so whole-frame
// tiles keep the query traffic near one read per frame; the channel slices
// give the grid enough workgroups.  Each slice of the query is streamed
// through LDS in chunks of 4 x 32 channels (double buffered, staged through
// registers), where all waves of the workgroup read it as their MFMA B
// operand.  X goes straight from HBM into A-operand registers with 16-byte
// buffer loads, one chunk ahead of use.  Per 32-channel step each wave runs
// v_mfma_f32_16x16x32_bf16 for
//     S += X Q^T      (the relevance contraction),
//     G += X X^T      (diagonal: |x|^2),
//     P += X I        (identity columns: the channel sums of its 16 tokens),
// so token norms and pooling cost no vector-ALU work (the threads that stage the
// query add up |q_j|^2 as they go).  Channel sums of the waves meet in LDS and
// are added in wave order once per chunk.
//
// With one slice a workgroup finishes its tokens' a_{t,n} itself; with several
// it writes its partial x . q_j and |x|^2.  The last workgroup of a frame
// (atomic counter) adds the partials in a fixed order: a_{t,n} (several
// slices), the pooled feature p_t, |p_t|^2 and r_t.  The second workgroup to
// finish of each adjacent pair (t-1, t) writes delta_t, evaluated as
// |p_t/|p_t| - p_{t-1}/|p_{t-1}||^2 / 2 (equal to 1 - cos, without its
// cancellation for nearly equal frames).  Nothing waits on a counter; each is
// reset by the workgroup that acts on it.
//
// Vector-ALU path (fp32 inputs, Q < 16 or tiny frames): tiles of up to 32
// tokens over all channels, one wave per token, wave-reduced dot products.
#include <type_traits>

#include "wz_internal.h"

namespace wz {
namespace {

constexpr int kKStep = 32;    // channels per MFMA K step (16x16x32)
constexpr int kQMax = 1024;   // validated bound on query tokens

// ---------------------------------------------------------------------------
// Memory helpers
// ---------------------------------------------------------------------------

// Buffer-resource accesses: an offset at or past the resource's size reads
// zeros / drops the write without touching memory, so pad rows and ragged
// edges need no branch (branches around loads would make the compiler wait
// for every outstanding load before each MFMA batch).
constexpr int kOOB = 0x40000000;       // byte offset beyond any resource here
constexpr int kBufWord3 = 0x00020000;  // gfx9-family raw buffer descriptor word 3
constexpr int kSc1 = 16;               // cache policy: device-scope coherent

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, int(bytes), kBufWord3);
}
__device__ __forceinline__ bf16x8 buf_load_bf16x8(__amdgpu_buffer_rsrc_t r, int off) {
  return __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
}
__device__ __forceinline__ u32x4 buf_load_u32x4(__amdgpu_buffer_rsrc_t r, int off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
}
__device__ __forceinline__ void buf_store_dev(float v, __amdgpu_buffer_rsrc_t r, int off) {
  __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v), r, off, 0, kSc1);
}

// Cross-workgroup data of this kernel is written with device-scope relaxed
// atomic stores (or sc1 buffer stores), which write through the XCD-local L2
// to the device's coherence point, and read back with device-scope relaxed
// atomic loads, which do not hit stale cache lines.  Ordering comes from
// waiting for a wave's stores to complete before the counter update that
// publishes them; no L2 writeback or invalidate is needed.
__device__ __forceinline__ void st_dev(float* p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_dev(double* p, double v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float ld_dev(const float* p) {
  return __hip_atomic_load(const_cast<float*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ double ld_dev(const double* p) {
  return __hip_atomic_load(const_cast<double*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float2 ld_dev2(const float* p) {
  const uint64_t u = __hip_atomic_load(reinterpret_cast<uint64_t*>(const_cast<float*>(p)), __ATOMIC_RELAXED,
                                       __HIP_MEMORY_SCOPE_AGENT);
  return make_float2(__uint_as_float(uint32_t(u)), __uint_as_float(uint32_t(u >> 32)));
}
__device__ __forceinline__ void st_dev2(float* p, float2 v) {
  const uint64_t u = uint64_t(__float_as_uint(v.x)) | (uint64_t(__float_as_uint(v.y)) << 32);
  __hip_atomic_store(reinterpret_cast<uint64_t*>(p), u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// Wait until this wave's memory operations have completed (compiler barriers
// keep the surrounding accesses on their side of the wait).
__device__ __forceinline__ void wait_memory() {
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  __builtin_amdgcn_s_waitcnt(0);
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
}
__device__ __forceinline__ int counter_add(int* p, int v) {
  return __hip_atomic_fetch_add(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Device-coherent (sc1) buffer loads of data other workgroups of this launch
// wrote; plain loads, so the compiler batches them freely.
__device__ __forceinline__ float ld_dev_buf(__amdgpu_buffer_rsrc_t r, int off) {
  return __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, off, 0, kSc1));
}
__device__ __forceinline__ f32x4 ld_dev_buf4(__amdgpu_buffer_rsrc_t r, int off) {
  return __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, kSc1));
}
__device__ __forceinline__ double ld_dev_buf_f64(__amdgpu_buffer_rsrc_t r, int off) {
  return __builtin_bit_cast(double, __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, kSc1));
}
__device__ __forceinline__ void buf_store_dev_f64(double v, __amdgpu_buffer_rsrc_t r, int off) {
  __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(uint32_t __attribute__((ext_vector_type(2))), v), r,
                                        off, 0, kSc1);
}

// Order-preserving map of floats onto unsigned integers (for exact maxima
// with integer LDS atomics): larger float <=> larger key; 0 is below every key.
__device__ __forceinline__ uint32_t max_key(float v) {
  const uint32_t u = __float_as_uint(v);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float key_value(uint32_t k) {
  return __uint_as_float((k & 0x80000000u) ? (k & 0x7fffffffu) : ~k);
}

// ---------------------------------------------------------------------------
// Block reductions (any multiple of 64 threads up to 1024)
// ---------------------------------------------------------------------------
__device__ double block_sum_f64(double v, double* s_red) {
  v = wave_sum_f64(v);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
  __syncthreads();
  if (lane == 0) s_red[wave] = v;
  __syncthreads();
  double s = 0.0;
  for (int i = 0; i < nw; ++i) s += s_red[i];
  return s;
}

__device__ double block_max_f64(double v, double* s_red) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v = fmax(v, __shfl_xor(v, m, kWave));
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
  __syncthreads();
  if (lane == 0) s_red[wave] = v;
  __syncthreads();
  double s = -INFINITY;
  for (int i = 0; i < nw; ++i) s = fmax(s, s_red[i]);
  return s;
}

// ---------------------------------------------------------------------------
// Finishing a frame and a pair of frames (run by the last workgroup of each)
// ---------------------------------------------------------------------------
struct FrameArgs {
  float* s_part;
  float* g_part;
  float* qg_part;
  float* sig_part;
  float* pool_part;
  double* pn2_part;
  Counters* ctr;
  float* tok_score;
  float* frame_rel;
  float* frame_delta;
  int T, N, C, Q, QP, tiles, slices;
};

// LDS of the finishing steps.
struct FinLds {
  float rq[kQMax];        // 1 / |q_j|
  float xn[kTokMax];      // |x_{t,n}| (several slices)
  uint32_t best[kTokMax]; // max_j of x . q_j / |q_j| as max_key (several slices)
  double red[3 * kMaxWaves];
  int flag[4];
};

// Frame t: a_{t,n} from the slices' partial dot products (several slices),
// |p_t|^2 and r_t.  L.rq holds 1/|q_j| when rq_local.  Every partial is added
// in index order (slice, then tile), so results do not depend on timing.
__device__ void frame_finish(const FrameArgs& f, int t, FinLds& L, bool rq_local) {
  const int tid = threadIdx.x, nthreads = blockDim.x;
  const int N = f.N, C = f.C, Q = f.Q, QP = f.QP, S = f.slices, tiles = f.tiles, K = tiles * S;
  const int G4 = QP / 4, units = N * G4;
  const __amdgpu_buffer_rsrc_t sres =
      make_rsrc(f.s_part + size_t(t) * S * N * QP, S > 1 ? uint32_t(S) * N * QP * 4 : 0u);
  const __amdgpu_buffer_rsrc_t qgres = make_rsrc(f.qg_part + size_t(t) * S * Q, rq_local ? 0u : uint32_t(S) * Q * 4);
  const __amdgpu_buffer_rsrc_t sgres = make_rsrc(f.sig_part + size_t(t) * K * Q, uint32_t(K) * Q * 4);
  const __amdgpu_buffer_rsrc_t gres = make_rsrc(f.g_part + size_t(t) * S * N, S > 1 ? uint32_t(S) * N * 4 : 0u);
  const __amdgpu_buffer_rsrc_t pnres = make_rsrc(f.pn2_part + size_t(t) * S, tiles == 1 ? uint32_t(S) * 8 : 0u);

  // first batch of partial dot products, in flight during the small sums below
  constexpr int U = 4, SB = 4;
  f32x4 v[U][SB];
  auto load_batch = [&](int u0, int s0) {
#pragma unroll
    for (int k = 0; k < U; ++k)
#pragma unroll
      for (int s = 0; s < SB; ++s) {
        const int u = u0 + tid + k * nthreads;
        const bool ok = u < units && s0 + s < S;
        v[k][s] = ld_dev_buf4(sres, ok ? ((s0 + s) * N * QP + u * 4) * 4 : kOOB);
      }
  };
  if (S > 1) load_batch(0, 0);

  // 1/|q_j|, sigma_j = sum over tokens of x . q_j, |x_n| (several slices), |p_t|^2
  double rbest = -INFINITY, pn2 = 0.0;
  for (int i = tid; i < max(Q, S > 1 ? N : 0); i += nthreads) {
    float qq = 0.f, sg = 0.f, xx = 0.f;
    double pp = 0.0;
    for (int k0 = 0; k0 < K; k0 += 4) {
      float a[4], b[4], c[4];
      double d[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int k = k0 + e;
        a[e] = ld_dev_buf(qgres, (i < Q && k < S) ? (k * Q + i) * 4 : kOOB);
        b[e] = ld_dev_buf(sgres, (i < Q && k < K) ? (k * Q + i) * 4 : kOOB);
        c[e] = ld_dev_buf(gres, (i < N && k < S) ? (k * N + i) * 4 : kOOB);
        d[e] = ld_dev_buf_f64(pnres, (i == 0 && k < S) ? k * 8 : kOOB);
      }
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        qq += a[e];
        sg += b[e];
        xx += c[e];
        pp += d[e];
      }
    }
    if (i < Q) {
      const float rq = rq_local ? L.rq[i] : (qq > 0.f ? 1.0f / sqrtf(qq) : 0.f);
      if (!rq_local) L.rq[i] = rq;
      rbest = fmax(rbest, double(sg) * rq);
    }
    if (S > 1 && i < N) {
      L.xn[i] = sqrtf(xx);
      L.best[i] = 0u;
    }
    if (i == 0) pn2 = pp;
  }
  if (tiles > 1) {
    // several token tiles: |p_t|^2 from the tiles' channel sums
    pn2 = 0.0;
    const __amdgpu_buffer_rsrc_t pres = make_rsrc(f.pool_part + size_t(t) * tiles * C, uint32_t(tiles) * C * 4);
    for (int c4 = tid; c4 < C / 4; c4 += nthreads) {
      f32x4 p = {0.f, 0.f, 0.f, 0.f};
      for (int k = 0; k < tiles; ++k) p += ld_dev_buf4(pres, (k * C + c4 * 4) * 4);
      pn2 += double(p[0]) * p[0] + double(p[1]) * p[1] + double(p[2]) * p[2] + double(p[3]) * p[3];
    }
  }
  pn2 = block_sum_f64(pn2, L.red);  // (its barrier also publishes L.rq / L.xn / L.best)
  rbest = block_max_f64(rbest, L.red);

  if (S > 1) {
    // a_{t,n} = max_j (sum_s S_s[n][j]) / |q_j| / |x_n|
    for (int u0 = 0; u0 < units; u0 += U * nthreads) {
      f32x4 acc[U];
#pragma unroll
      for (int k = 0; k < U; ++k) acc[k] = f32x4{0.f, 0.f, 0.f, 0.f};
      for (int s0 = 0; s0 < S; s0 += SB) {
        if (u0 > 0 || s0 > 0) load_batch(u0, s0);
#pragma unroll
        for (int k = 0; k < U; ++k)
#pragma unroll
          for (int s = 0; s < SB; ++s) acc[k] += v[k][s];
      }
#pragma unroll
      for (int k = 0; k < U; ++k) {
        const int u = u0 + tid + k * nthreads;
        if (u < units) {
          const int n = u / G4, j0 = (u % G4) * 4;
          float m = -INFINITY;
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (j0 + e < Q) m = fmaxf(m, acc[k][e] * L.rq[j0 + e]);
          if (j0 < Q) atomicMax(&L.best[n], max_key(m));
        }
      }
    }
    __syncthreads();
    for (int n = tid; n < N; n += nthreads) {
      const float xn = L.xn[n];
      f.tok_score[size_t(t) * N + n] = xn > 0.f ? key_value(L.best[n]) / xn : 0.f;
    }
  }
  if (tid == 0) {
    const double pn = sqrt(pn2);
    f.frame_rel[t] = float(pn > 0.0 ? rbest / pn : 0.0);
    if (t == 0) f.frame_delta[0] = 0.f;
    __hip_atomic_store(&f.ctr->frame[t], 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

// delta_p = clamp(1 - cos(p_p, p_{p-1}), 0, 2) from the two frames' channel
// sums (tile partials added in tile order); a zero vector gives delta = 1.
__device__ void pair_finish(const FrameArgs& f, int p, FinLds& L) {
  const int tid = threadIdx.x, nthreads = blockDim.x, C = f.C, tiles = f.tiles, C4 = C / 4;
  const __amdgpu_buffer_rsrc_t ares = make_rsrc(f.pool_part + size_t(p - 1) * tiles * C, uint32_t(tiles) * C * 4);
  const __amdgpu_buffer_rsrc_t bres = make_rsrc(f.pool_part + size_t(p) * tiles * C, uint32_t(tiles) * C * 4);
  double ab = 0.0, aa = 0.0, bb = 0.0;
  for (int c0 = tid; c0 < C4; c0 += 2 * nthreads) {
    f32x4 a[2], b[2];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int c4 = c0 + h * nthreads;
      a[h] = ld_dev_buf4(ares, c4 < C4 ? c4 * 16 : kOOB);
      b[h] = ld_dev_buf4(bres, c4 < C4 ? c4 * 16 : kOOB);
    }
    for (int k = 1; k < tiles; ++k) {
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int c4 = c0 + h * nthreads;
        a[h] += ld_dev_buf4(ares, c4 < C4 ? (k * C + c4 * 4) * 4 : kOOB);
        b[h] += ld_dev_buf4(bres, c4 < C4 ? (k * C + c4 * 4) * 4 : kOOB);
      }
    }
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        ab += double(a[h][e]) * b[h][e];
        aa += double(a[h][e]) * a[h][e];
        bb += double(b[h][e]) * b[h][e];
      }
  }
  ab = wave_sum_f64(ab);
  aa = wave_sum_f64(aa);
  bb = wave_sum_f64(bb);
  const int lane = tid & 63, wave = tid >> 6, nw = nthreads >> 6;
  __syncthreads();
  if (lane == 0) {
    L.red[3 * wave] = ab;
    L.red[3 * wave + 1] = aa;
    L.red[3 * wave + 2] = bb;
  }
  __syncthreads();
  if (tid == 0) {
    double sab = 0.0, saa = 0.0, sbb = 0.0;
    for (int w = 0; w < nw; ++w) {
      sab += L.red[3 * w];
      saa += L.red[3 * w + 1];
      sbb += L.red[3 * w + 2];
    }
    double delta = 1.0;
    if (saa > 0.0 && sbb > 0.0) delta = fmin(fmax(1.0 - sab / sqrt(saa * sbb), 0.0), 2.0);
    f.frame_delta[p] = float(delta);
    __hip_atomic_store(&f.ctr->pair[p], 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

// Called by every workgroup once its unit's sums are written: counts the unit
// for its frame and for the two pairs the frame belongs to, and runs the
// finishing step of each one it completes.
__device__ void unit_finished(const FrameArgs& f, int t, FinLds& L, bool rq_local) {
  const int tid = threadIdx.x;
  const int units = f.tiles * f.slices;
  wait_memory();
  __syncthreads();
  if (tid == 0) {
    // pair[p] counts the units of frames p-1 and p; frame 0 adds nothing to
    // pair[0] and frame T-1 nothing to pair[T]
    const int c0 = counter_add(&f.ctr->frame[t], 1);
    const int c1 = counter_add(&f.ctr->pair[t], t >= 1 ? 1 : 0);
    const int c2 = counter_add(&f.ctr->pair[t + 1], t + 1 < f.T ? 1 : 0);
    L.flag[0] = c0 == units - 1;
    L.flag[1] = t >= 1 && c1 == 2 * units - 1;
    L.flag[2] = t + 1 < f.T && c2 == 2 * units - 1;
  }
  __syncthreads();
  const bool fin = L.flag[0], p0 = L.flag[1], p1 = L.flag[2];
  if (fin) frame_finish(f, t, L, rq_local);
  if (p0) pair_finish(f, t, L);
  if (p1) pair_finish(f, t + 1, L);
}

// ---------------------------------------------------------------------------
// MFMA path
// ---------------------------------------------------------------------------
// NTG: 16-column query tiles per pass over the slice (queries of more tokens
// take several passes); R: depth of the X prefetch ring in 32-channel steps.
template <int NTG, int R>
__global__ __launch_bounds__(kMaxWaves / kTilesPerWave * 64) void k_relevance_mfma(const uint16_t* __restrict__ X,
                                                                                   const uint16_t* __restrict__ query,
                                                                                   int tile_tokens, int kc,
                                                                                   FrameArgs f) {
  constexpr int MTW = kTilesPerWave;
  constexpr int MAXW = kMaxWaves / MTW;
  constexpr int QB = 8;                          // query units staged per thread per batch
  __shared__ u32x4 s_q[kSliceSteps][NTG][kWave];  // the group's query slice, MFMA B layout
  __shared__ float s_poolw[MAXW][kSliceSteps * kKStep];  // per-wave channel sums of the slice
  __shared__ float s_colw[MAXW][NTG * 16];       // per-wave column sums of S
  __shared__ float s_qgw[MAXW][NTG * 16];        // per-wave |q_j|^2 partials
  __shared__ float s_xt[kMaxWaves * 16];         // |x| of the tile's tokens (one slice)
  __shared__ FinLds L;

  int t, tile, sl;
  unit_of_block(blockIdx.x, f.tiles, f.slices, t, tile, sl);
  if (t >= f.T) return;
  const int N = f.N, C = f.C, Q = f.Q, QP = f.QP, S = f.slices;
  const int tok0 = tile * tile_tokens;
  const int TM = min(tile_tokens, N - tok0);
  const int tid = threadIdx.x, nthreads = blockDim.x;
  // wave index in a scalar register: branches on it must be scalar branches,
  // since an MFMA under an exec mask still updates every lane
  const int lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6), nw = nthreads >> 6;
  const int row = lane & 15, grp = lane >> 4;
  const int c_lo = sl * kc, c_hi = min(C, c_lo + kc);
  const int kper = (c_hi - c_lo + kKStep - 1) / kKStep;  // <= kSliceSteps

  const __amdgpu_buffer_rsrc_t xres = make_rsrc(X + (size_t(t) * N + tok0) * C, uint32_t(TM) * C * 2);
  const __amdgpu_buffer_rsrc_t qres = make_rsrc(query, uint32_t(Q) * C * 2);
  int xoff[MTW];  // byte offsets of this lane's token rows (A operands) in the tile
#pragma unroll
  for (int i = 0; i < MTW; ++i) {
    const int r = (wave * MTW + i) * 16 + row;
    xoff[i] = r < TM ? r * C * 2 : kOOB;
  }

  // identity operands: slot e of the lane with column `row`, K group `grp`
  // holds channel 8*grp + e of the step; I_s selects channel 16*s + column
  bf16x8 I0, I1;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    I0[e] = (__bf16)((8 * grp + e == row) ? 1.0f : 0.0f);
    I1[e] = (__bf16)((8 * grp + e == 16 + row) ? 1.0f : 0.0f);
  }

  f32x4 G[MTW];
  float best[MTW][4];  // rows 16*(wave*MTW+i) + 4*grp + e (one slice only)
#pragma unroll
  for (int i = 0; i < MTW; ++i) {
    G[i] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int e = 0; e < 4; ++e) best[i][e] = -INFINITY;
  }
  const int groups = (Q + NTG * 16 - 1) / (NTG * 16);

  bf16x8 a[R][MTW];  // X prefetch ring: slot r holds the steps ks = r (mod R)
  auto issue = [&](int ks, bf16x8 (&dst)[MTW]) {
    const int c = c_lo + ks * kKStep + grp * 8;
    const bool ok = ks < kper && c < c_hi;
#pragma unroll
    for (int i = 0; i < MTW; ++i) dst[i] = buf_load_bf16x8(xres, ok ? xoff[i] + c * 2 : kOOB);
  };

  for (int g = 0; g < groups; ++g) {
    const int qg0 = g * NTG * 16;
    f32x4 Sacc[MTW][NTG], QG[NTG];
#pragma unroll
    for (int n = 0; n < NTG; ++n) {
      QG[n] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int i = 0; i < MTW; ++i) Sacc[i][n] = f32x4{0.f, 0.f, 0.f, 0.f};
    }

    // X ring first, then the query slice of the group into LDS: unit
    // u -> step u / (64 NTG), tile (u / 64) % NTG, lane u % 64
#pragma unroll
    for (int r = 0; r < R; ++r) issue(r, a[r]);
    const int qunits = kper * NTG * kWave;
    for (int u0 = 0; u0 < qunits; u0 += QB * nthreads) {
      u32x4 qv[QB];
#pragma unroll
      for (int k = 0; k < QB; ++k) {
        const int u = u0 + tid + k * nthreads;
        const int l = u & 63, n = (u >> 6) % NTG, ks = u / (NTG * kWave);
        const int j = qg0 + n * 16 + (l & 15);
        const int c = c_lo + ks * kKStep + (l >> 4) * 8;
        const bool ok = u < qunits && j < Q && c < c_hi;
        qv[k] = buf_load_u32x4(qres, ok ? (j * C + c) * 2 : kOOB);
      }
#pragma unroll
      for (int k = 0; k < QB; ++k) {
        const int u = u0 + tid + k * nthreads;
        if (u < qunits) s_q[u / (NTG * kWave)][(u >> 6) % NTG][u & 63] = qv[k];
      }
    }
    __syncthreads();

    auto compute = [&](int ks, const bf16x8 (&x)[MTW], auto pool) {
      bf16x8 b[NTG];
#pragma unroll
      for (int n = 0; n < NTG; ++n) b[n] = __builtin_bit_cast(bf16x8, s_q[ks][n][lane]);
#pragma unroll
      for (int n = 0; n < NTG; ++n)
#pragma unroll
        for (int i = 0; i < MTW; ++i)
          Sacc[i][n] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(x[i], b[n], Sacc[i][n], 0, 0, 0);
      if (ks % nw == wave) {
        // query Gram matrix of the step (diagonal: |q_j|^2), spread over the waves
#pragma unroll
        for (int n = 0; n < NTG; ++n) QG[n] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(b[n], b[n], QG[n], 0, 0, 0);
      }
      if constexpr (decltype(pool)::value) {
        f32x4 P0 = {0.f, 0.f, 0.f, 0.f}, P1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int i = 0; i < MTW; ++i) {
          G[i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(x[i], x[i], G[i], 0, 0, 0);
          P0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(x[i], I0, P0, 0, 0, 0);
          P1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(x[i], I1, P1, 0, 0, 0);
        }
        float v0 = (P0[0] + P0[1]) + (P0[2] + P0[3]);
        float v1 = (P1[0] + P1[1]) + (P1[2] + P1[3]);
        v0 += __shfl_xor(v0, 16, kWave);
        v1 += __shfl_xor(v1, 16, kWave);
        v0 += __shfl_xor(v0, 32, kWave);
        v1 += __shfl_xor(v1, 32, kWave);
        // lanes 0-15: channels 32ks+0..15 of the slice, lanes 16-31: 32ks+16..31
        if (lane < 32) s_poolw[wave][ks * kKStep + lane] = lane < 16 ? v0 : v1;
      }
    };
    auto run = [&](auto pool) {
      for (int ks0 = 0; ks0 < kper; ks0 += R) {
#pragma unroll
        for (int r = 0; r < R; ++r) {
          const int ks = ks0 + r;
          if (ks < kper) compute(ks, a[r], pool);
          issue(ks + R, a[r]);
        }
      }
    };
    if (g == 0) run(std::true_type{});
    else run(std::false_type{});
    __syncthreads();

    // ---- group epilogue ----
    const bool diag = (row >> 2) == grp;  // lane holds element (row, row) of a 16x16 tile
    if (diag) {
#pragma unroll
      for (int n = 0; n < NTG; ++n) s_qgw[wave][n * 16 + row] = QG[n][row & 3];
    }
#pragma unroll
    for (int n = 0; n < NTG; ++n) {
      float v = 0.f;
#pragma unroll
      for (int i = 0; i < MTW; ++i) v += (Sacc[i][n][0] + Sacc[i][n][1]) + (Sacc[i][n][2] + Sacc[i][n][3]);
      v += __shfl_xor(v, 16, kWave);
      v += __shfl_xor(v, 32, kWave);
      if (lane < 16) s_colw[wave][n * 16 + lane] = v;
    }
    if (g == 0) {
      const __amdgpu_buffer_rsrc_t gres = make_rsrc(f.g_part + (size_t(t) * S + sl) * N, S > 1 ? uint32_t(N) * 4 : 0u);
      if (diag) {
#pragma unroll
        for (int i = 0; i < MTW; ++i) {
          const int r = (wave * MTW + i) * 16 + row;
          const float gg = G[i][row & 3];
          if (S == 1) s_xt[r] = sqrtf(gg);
          else buf_store_dev(gg, gres, r < TM ? (tok0 + r) * 4 : kOOB);
        }
      }
      // the slice's channel sums, waves added in order; their squares for |p_t|^2
      const __amdgpu_buffer_rsrc_t pres =
          make_rsrc(f.pool_part + (size_t(t) * f.tiles + tile) * C, uint32_t(C) * 4);
      double pp = 0.0;
      for (int c = tid; c < kper * kKStep; c += nthreads) {
        float s = 0.f;
        for (int w = 0; w < nw; ++w) s += s_poolw[w][c];
        const bool in = c_lo + c < c_hi;
        buf_store_dev(s, pres, in ? (c_lo + c) * 4 : kOOB);
        if (in) pp += double(s) * s;
      }
      if (f.tiles == 1) {
        pp = block_sum_f64(pp, L.red);
        if (tid == 0) st_dev(f.pn2_part + size_t(t) * S + sl, pp);
      }
    }
    __syncthreads();
    if (tid < NTG * 16) {
      const int j = qg0 + tid;
      float qq = 0.f, sg = 0.f;
      for (int w = 0; w < nw; ++w) {
        qq += s_qgw[w][tid];
        sg += s_colw[w][tid];
      }
      if (j < Q) {
        if (S == 1) L.rq[j] = qq > 0.f ? 1.0f / sqrtf(qq) : 0.f;
        else if (tile == 0) st_dev(f.qg_part + (size_t(t) * S + sl) * Q + j, qq);
        st_dev(f.sig_part + ((size_t(t) * f.tiles + tile) * S + sl) * Q + j, sg);
      }
    }
    __syncthreads();
    const __amdgpu_buffer_rsrc_t sres =
        make_rsrc(f.s_part + (size_t(t) * S + sl) * N * QP, S > 1 ? uint32_t(N) * QP * 4 : 0u);
#pragma unroll
    for (int n = 0; n < NTG; ++n) {
      const int j = qg0 + n * 16 + row;  // this lane's column
      if (S == 1) {
        const float rq = j < Q ? L.rq[j] : 0.f;
#pragma unroll
        for (int i = 0; i < MTW; ++i)
#pragma unroll
          for (int e = 0; e < 4; ++e) best[i][e] = fmaxf(best[i][e], j < Q ? Sacc[i][n][e] * rq : -INFINITY);
      } else {
#pragma unroll
        for (int i = 0; i < MTW; ++i)
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int r = (wave * MTW + i) * 16 + 4 * grp + e;
            buf_store_dev(Sacc[i][n][e], sres, (r < TM && j < Q) ? ((tok0 + r) * QP + j) * 4 : kOOB);
          }
      }
    }
  }

  if (S == 1) {
    // max over the 16 columns held by the lanes of this K group
#pragma unroll
    for (int i = 0; i < MTW; ++i)
#pragma unroll
      for (int e = 0; e < 4; ++e)
#pragma unroll
        for (int m = 1; m < 16; m <<= 1) best[i][e] = fmaxf(best[i][e], __shfl_xor(best[i][e], m, kWave));
    if (row == 0) {
#pragma unroll
      for (int i = 0; i < MTW; ++i)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int r = (wave * MTW + i) * 16 + 4 * grp + e;
          if (r < TM) {
            const float xn = s_xt[r];
            f.tok_score[size_t(t) * N + tok0 + r] = xn > 0.f ? best[i][e] / xn : 0.f;
          }
        }
    }
  }
  unit_finished(f, t, L, S == 1);
}

// ---------------------------------------------------------------------------
// Vector-ALU path
// ---------------------------------------------------------------------------
template <typename In>
struct Vec;
template <>
struct Vec<float> {
  static constexpr int kN = 4;
  __device__ static void load(const float* p, float* v) {
    const f32x4 x = *reinterpret_cast<const f32x4*>(p);
    v[0] = x[0]; v[1] = x[1]; v[2] = x[2]; v[3] = x[3];
  }
};
template <>
struct Vec<uint16_t> {
  static constexpr int kN = 8;
  __device__ static void load(const uint16_t* p, float* v) {
    const u32x4 x = *reinterpret_cast<const u32x4*>(p);
#pragma unroll
    for (int i = 0; i < 4; ++i) { v[2 * i] = bf16_lo(x[i]); v[2 * i + 1] = bf16_hi(x[i]); }
  }
};

template <typename In>
__global__ __launch_bounds__(256) void k_relevance_valu(const In* __restrict__ X, const In* __restrict__ query,
                                                        int tile_tokens, FrameArgs f) {
  constexpr int NW = 4;
  constexpr int V = Vec<In>::kN;
  constexpr int QB = 16;
  __shared__ float s_sig[NW][kQMax];
  __shared__ FinLds L;
  float* s_rq = L.rq;

  int t, tile, sl;
  unit_of_block(blockIdx.x, f.tiles, 1, t, tile, sl);
  if (t >= f.T) return;
  const int N = f.N, C = f.C, Q = f.Q;
  const int tok0 = tile * tile_tokens;
  const int TM = min(tile_tokens, N - tok0);
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int nvec = C / V;
  const size_t part = size_t(t) * f.tiles + tile;

  // 1 / |q_j|
  for (int j = wave; j < Q; j += NW) {
    float s = 0.f;
    for (int v = lane; v < nvec; v += kWave) {
      float q[V];
      Vec<In>::load(query + size_t(j) * C + v * V, q);
#pragma unroll
      for (int i = 0; i < V; ++i) s += q[i] * q[i];
    }
    s = wave_sum(s);
    if (lane == 0) s_rq[j] = s > 0.f ? 1.0f / sqrtf(s) : 0.f;
  }
  for (int j = tid; j < NW * kQMax; j += 256) (&s_sig[0][0])[j] = 0.f;
  __syncthreads();

  for (int r = wave; r < TM; r += NW) {
    const In* x = X + (size_t(t) * N + tok0 + r) * C;
    float best = -INFINITY, xn2 = 0.f;
    for (int j0 = 0; j0 < Q; j0 += QB) {
      float d[QB];
#pragma unroll
      for (int k = 0; k < QB; ++k) d[k] = 0.f;
      float n2 = 0.f;
      for (int v = lane; v < nvec; v += kWave) {
        float xv[V];
        Vec<In>::load(x + v * V, xv);
#pragma unroll
        for (int i = 0; i < V; ++i) n2 += xv[i] * xv[i];
#pragma unroll
        for (int k = 0; k < QB; ++k) {
          if (j0 + k < Q) {
            float qv[V];
            Vec<In>::load(query + size_t(j0 + k) * C + v * V, qv);
#pragma unroll
            for (int i = 0; i < V; ++i) d[k] += xv[i] * qv[i];
          }
        }
      }
      if (j0 == 0) xn2 = wave_sum(n2);
#pragma unroll
      for (int k = 0; k < QB; ++k) {
        if (j0 + k < Q) {
          const float s = wave_sum(d[k]);
          best = fmaxf(best, s * s_rq[j0 + k]);
          if (lane == 0) s_sig[wave][j0 + k] += s;
        }
      }
    }
    if (lane == 0) {
      const float xn = sqrtf(xn2);
      f.tok_score[size_t(t) * N + tok0 + r] = xn > 0.f ? best / xn : 0.f;
    }
  }

  // channel sums of the tile (tokens in order); with one tile, |p_t|^2
  double pp = 0.0;
  for (int v = tid; v < nvec; v += 256) {
    float acc[V];
#pragma unroll
    for (int i = 0; i < V; ++i) acc[i] = 0.f;
    for (int r = 0; r < TM; ++r) {
      float xv[V];
      Vec<In>::load(X + (size_t(t) * N + tok0 + r) * C + v * V, xv);
#pragma unroll
      for (int i = 0; i < V; ++i) acc[i] += xv[i];
    }
#pragma unroll
    for (int i = 0; i < V; ++i) {
      st_dev(f.pool_part + part * C + v * V + i, acc[i]);
      pp += double(acc[i]) * acc[i];
    }
  }
  if (f.tiles == 1) {
    pp = block_sum_f64(pp, L.red);
    if (tid == 0) st_dev(f.pn2_part + t, pp);
  }
  __syncthreads();
  for (int j = tid; j < Q; j += 256) {
    float s = 0.f;
    for (int w = 0; w < NW; ++w) s += s_sig[w][j];
    st_dev(f.sig_part + part * Q + j, s);
  }
  unit_finished(f, t, L, true);
}

#ifndef WZ_REL_RING
#define WZ_REL_RING 8  // X prefetch depth in 32-channel steps
#endif

template <int NTG>
void launch_mfma(const RelPlan& pl, const void* X, const void* query, const FrameArgs& fa, hipStream_t s) {
  hipLaunchKernelGGL((k_relevance_mfma<NTG, WZ_REL_RING>), dim3(pl.grid), dim3(pl.threads), 0, s,
                     static_cast<const uint16_t*>(X), static_cast<const uint16_t*>(query), pl.tile_tokens, pl.kc,
                     fa);
}

}  // namespace

bool relevance_uses_mfma(const wz_config& c) {
  // two 16-row MFMA tiles per wave, at least 2 waves: frames of at least 49 tokens
  return c.in_dtype == WZ_BF16 && c.Q >= 16 && c.H * c.W >= 49;
}

hipError_t launch_relevance(const wz_config& c, const void* X, const void* query, float* tok_score,
                            float* frame_rel, float* frame_delta, const Workspace& ws, hipStream_t s) {
  const RelPlan pl = relevance_plan(c);
  FrameArgs fa{ws.s_part, ws.g_part,  ws.qg_part,  ws.sig_part,  ws.pool_part, ws.pn2_part, ws.ctr,
               tok_score, frame_rel, frame_delta, c.T,          c.H * c.W,    c.C,          c.Q,
               qpad(c.Q),  pl.tiles,   pl.slices};
  if (relevance_uses_mfma(c)) {
    // queries of more than 32 tokens take several passes of 32 over the slice:
    // wider query groups no longer fit the accumulators in registers
    if (c.Q <= 16) launch_mfma<1>(pl, X, query, fa, s);
    else launch_mfma<2>(pl, X, query, fa, s);
  } else if (c.in_dtype == WZ_BF16) {
    hipLaunchKernelGGL((k_relevance_valu<uint16_t>), dim3(pl.grid), dim3(pl.threads), 0, s,
                       static_cast<const uint16_t*>(X), static_cast<const uint16_t*>(query), pl.tile_tokens, fa);
  } else {
    hipLaunchKernelGGL((k_relevance_valu<float>), dim3(pl.grid), dim3(pl.threads), 0, s,
                       static_cast<const float*>(X), static_cast<const float*>(query), pl.tile_tokens, fa);
  }
  return hipGetLastError();
}

}  // namespace wz
