// Stage 1: similarity-branch Cross-Modal Scorer (Sec. 3.2.1) and Visual Change
// Estimator (Sec. 3.2.2, Eq. (8)) in ONE kernel that streams the frames once.
//
// Every workgroup owns a tile of up to 32 consecutive tokens of one frame and
// reads all channels of them exactly once from HBM.  Per token it writes the
// saliency
//     a_{t,n} = max_j (x . q_j) / (|x| |q_j|)
// and, per tile, the channel sums and the sums of x . q_j over its tokens.
// The last workgroup to finish a frame (an atomic tile counter) combines the
// frame's tile sums in tile order into the pooled feature p_t = sum_n x_{t,n}
// and its norm, and writes the frame relevance
//     r_t = max_j (p_t . q_j) / (|p_t| |q_j|)      (the mean's cosine is the sum's).
// The last of the two workgroups finishing frames t-1 and t (a pair counter)
// writes the visual change
//     delta_t = clamp(1 - cos(p_t, p_{t-1}), 0, 2),  delta_0 = 0,
// evaluated as |p_t/|p_t| - p_{t-1}/|p_{t-1}||^2 / 2 (the same value without
// the cancellation of 1 - cos for nearly equal frames); cos := 0, so
// delta = 1, if a pooled feature is zero.  Nothing ever waits on a counter;
// each counter is reset by the workgroup that acts on it.
//
// MFMA path (bf16, Q >= 16): the relevance contraction S = X Q^T runs on
// v_mfma_f32_16x16x32_bf16.  A lane's 16-byte load of 8 consecutive channels
// of one token is already its A operand; the same registers also feed a Gram
// tile X X^T (its diagonal is |x|^2) and an identity tile X I (it adds the
// tile's tokens channel by channel, i.e. the pooled sum), so norms and pooling
// cost no vector-ALU work.  Each wave owns a contiguous run of 32-channel
// steps; the waves' partial results are combined through LDS in a fixed order.
//
// Vector-ALU path (fp32 inputs, or bf16 with Q < 16): one wave per token,
// lanes over 16-byte channel vectors, wave-reduced dot products.
#include <type_traits>

#include "wz_internal.h"

namespace wz {
namespace {

constexpr int kKStep = 32;    // channels per MFMA K step (16x16x32)
constexpr int kQMax = 1024;   // validated bound on query tokens
constexpr int kThreads = 256; // both relevance kernels run 4 waves

// Buffer-resource loads: an offset at or past the resource's size returns
// zeros without touching memory, so pad rows, channels past C and steps past
// a wave's range need no branch (branches around loads would force the
// compiler to wait for every outstanding load before each MFMA batch).
constexpr int kOOB = 0x40000000;         // byte offset beyond any resource here
constexpr int kBufWord3 = 0x00020000;    // gfx9-family raw buffer descriptor word 3
constexpr int kSc1 = 16;                 // cache policy: device-scope coherent

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, int(bytes), kBufWord3);
}
__device__ __forceinline__ bf16x8 buf_load_bf16x8(__amdgpu_buffer_rsrc_t r, int off) {
  return __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
}

// Cross-workgroup data of this kernel (tile sums, pooled features, norms) is
// written with device-scope relaxed atomic stores, which write through the
// XCD-local L2 to the device's coherence point, and read back with
// device-scope relaxed atomic loads, which do not hit stale cache lines.
// Ordering comes from waiting for a wave's stores to complete before the
// counter update that publishes them; no L2 writeback or invalidate is needed.
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
// Two consecutive floats as one 8-byte device-coherent access.
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

struct FrameArgs {
  float* pool_part;
  float* sig_part;
  float* pooled;
  double* pnorm2;
  Counters* ctr;
  float* frame_rel;
  float* frame_delta;
  int T, C, Q, tiles;
};

__device__ double block_sum_f64(double v, double* s_red) {
  v = wave_sum_f64(v);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) s_red[wave] = v;
  __syncthreads();
  return (s_red[0] + s_red[1]) + (s_red[2] + s_red[3]);
}

__device__ double block_max_f64(double v, double* s_red) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v = fmax(v, __shfl_xor(v, m, kWave));
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) s_red[wave] = v;
  __syncthreads();
  return fmax(fmax(s_red[0], s_red[1]), fmax(s_red[2], s_red[3]));
}

// Called by every workgroup after its tile's sums are written.  The last
// workgroup of frame t finishes the frame, then the pair(s) it completes.
// s_rq holds 1/|q_j| for all Q query tokens.
__device__ void tile_finished(const FrameArgs& f, int t, const float* s_rq, double* s_red, int* s_flag) {
  const int tid = threadIdx.x;
  wait_memory();
  __syncthreads();
  if (tid == 0) s_flag[0] = counter_add(&f.ctr->frame[t], 1) == f.tiles - 1;
  __syncthreads();
  if (!s_flag[0]) return;

  // pooled feature of frame t, tile sums added in tile order.  Channels go in
  // pairs (8-byte coherent loads); a thread keeps CB pairs x TB tiles of loads
  // in flight before adding them, so the frame costs one or two round trips.
  constexpr int CB = 4, TB = 8;
  const int C = f.C, tiles = f.tiles, C2 = f.C / 2;
  const float* part = f.pool_part + size_t(t) * tiles * C;
  double acc = 0.0;
  for (int c0 = tid; c0 < C2; c0 += kThreads * CB) {
    float2 sum[CB];
#pragma unroll
    for (int i = 0; i < CB; ++i) sum[i] = make_float2(0.f, 0.f);
    for (int k0 = 0; k0 < tiles; k0 += TB) {
      float2 v[CB][TB];
#pragma unroll
      for (int i = 0; i < CB; ++i)
#pragma unroll
        for (int kk = 0; kk < TB; ++kk) {
          const int c2 = c0 + i * kThreads, k = k0 + kk;
          v[i][kk] = (c2 < C2 && k < tiles) ? ld_dev2(part + size_t(k) * C + 2 * c2) : make_float2(0.f, 0.f);
        }
#pragma unroll
      for (int i = 0; i < CB; ++i)
#pragma unroll
        for (int kk = 0; kk < TB; ++kk)
          if (k0 + kk < tiles) { sum[i].x += v[i][kk].x; sum[i].y += v[i][kk].y; }
    }
#pragma unroll
    for (int i = 0; i < CB; ++i) {
      const int c2 = c0 + i * kThreads;
      if (c2 < C2) {
        st_dev2(f.pooled + size_t(t) * C + 2 * c2, sum[i]);
        acc += double(sum[i].x) * sum[i].x + double(sum[i].y) * sum[i].y;
      }
    }
  }
  double best = -INFINITY;
  for (int j = tid; j < f.Q; j += kThreads) {
    float s = 0.f;
    for (int k0 = 0; k0 < tiles; k0 += TB) {
      float v[TB];
#pragma unroll
      for (int kk = 0; kk < TB; ++kk)
        v[kk] = k0 + kk < tiles ? ld_dev(f.sig_part + (size_t(t) * tiles + k0 + kk) * f.Q + j) : 0.f;
#pragma unroll
      for (int kk = 0; kk < TB; ++kk)
        if (k0 + kk < tiles) s += v[kk];
    }
    best = fmax(best, double(s) * s_rq[j]);  // divided by |p_t| below
  }
  acc = block_sum_f64(acc, s_red);
  const double pn = sqrt(acc);
  best = block_max_f64(best, s_red);
  best = pn > 0.0 ? best / pn : 0.0;
  if (tid == 0) {
    st_dev(f.pnorm2 + t, acc);
    f.frame_rel[t] = float(best);
    if (t == 0) f.frame_delta[0] = 0.f;
    __hip_atomic_store(&f.ctr->frame[t], 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }

  // pairs (t-1, t) and (t, t+1): the second frame to finish computes delta
  wait_memory();
  __syncthreads();
  if (tid == 0) {
    s_flag[1] = t >= 1 && counter_add(&f.ctr->pair[t], 1) == 1;
    s_flag[2] = t + 1 < f.T && counter_add(&f.ctr->pair[t + 1], 1) == 1;
  }
  __syncthreads();
  for (int side = 0; side < 2; ++side) {
    if (!s_flag[1 + side]) continue;
    const int p = t + side;  // delta_p from frames p-1 and p
    const double na = sqrt(ld_dev(f.pnorm2 + p)), nb = sqrt(ld_dev(f.pnorm2 + p - 1));
    double delta = 1.0;
    if (na > 0.0 && nb > 0.0) {
      const float* a = f.pooled + size_t(p) * C;
      const float* b = f.pooled + size_t(p - 1) * C;
      double dd = 0.0;
      for (int c0 = tid; c0 < C2; c0 += kThreads * CB) {
        float2 va[CB], vb[CB];
#pragma unroll
        for (int i = 0; i < CB; ++i) {
          const int c2 = c0 + i * kThreads;
          va[i] = c2 < C2 ? ld_dev2(a + 2 * c2) : make_float2(0.f, 0.f);
          vb[i] = c2 < C2 ? ld_dev2(b + 2 * c2) : make_float2(0.f, 0.f);
        }
#pragma unroll
        for (int i = 0; i < CB; ++i) {
          const double dx = double(va[i].x) / na - double(vb[i].x) / nb;
          const double dy = double(va[i].y) / na - double(vb[i].y) / nb;
          dd += dx * dx + dy * dy;
        }
      }
      dd = block_sum_f64(dd, s_red);
      delta = fmin(fmax(0.5 * dd, 0.0), 2.0);
    }
    if (tid == 0) {
      f.frame_delta[p] = float(delta);
      __hip_atomic_store(&f.ctr->pair[p], 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
}

// MT: 16-row MFMA tiles per workgroup tile; NTG: 16-column query tiles per
// pass over the tile's channels; U: channel steps per register buffer.
template <int MT, int NTG, int U>
__global__ __launch_bounds__(kThreads) void k_relevance_mfma(const uint16_t* __restrict__ X,
                                                             const uint16_t* __restrict__ query, int N,
                                                             int tile_tokens, float* __restrict__ tok_score,
                                                             float* __restrict__ rq_out, FrameArgs f) {
  constexpr int NW = kThreads / kWave;
  constexpr int ROWS = MT * 16;
  constexpr int COLS = NTG * 16;
  __shared__ float s_red[NW][ROWS][17];
  __shared__ float s_gpart[NW][ROWS];
  __shared__ float s_qpart[NW][COLS];
  __shared__ float s_rq[kQMax];
  __shared__ float s_xn[ROWS];
  __shared__ double s_dred[NW];
  __shared__ int s_flag[4];

  int t, tile;
  tile_of_block(blockIdx.x, f.tiles, t, tile);
  if (t >= f.T) return;
  const int C = f.C, Q = f.Q;
  const int tok0 = tile * tile_tokens;
  const int TM = min(tile_tokens, N - tok0);
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int row = lane & 15;
  const int grp = lane >> 4;
  const int ksteps = (C + kKStep - 1) / kKStep;
  const int kper = (ksteps + NW - 1) / NW;           // contiguous channel steps per wave
  const int k_begin = wave * kper, k_end = min(ksteps, k_begin + kper);
  const size_t part = size_t(t) * f.tiles + tile;
  float* pool_part = f.pool_part;
  float* sig_part = f.sig_part;

  // Identity operands: slot i of the lane with column `row`, K group `grp`
  // holds channel 8*grp + i of the step; I_s selects channel 16*s + column.
  bf16x8 I0, I1;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    I0[i] = (__bf16)((8 * grp + i == row) ? 1.0f : 0.0f);
    I1[i] = (__bf16)((8 * grp + i == 16 + row) ? 1.0f : 0.0f);
  }

  // Byte offsets of this lane's token rows inside the tile's buffer resource.
  const __amdgpu_buffer_rsrc_t xres = make_rsrc(X + (size_t(t) * N + tok0) * C, uint32_t(TM) * C * 2);
  const __amdgpu_buffer_rsrc_t pres = make_rsrc(pool_part + part * C, uint32_t(C) * 4);
  int xoff[MT];
#pragma unroll
  for (int m = 0; m < MT; ++m) {
    const int r = m * 16 + row;
    xoff[m] = r < TM ? r * C * 2 : kOOB;
  }

  f32x4 G[MT];
#pragma unroll
  for (int m = 0; m < MT; ++m) G[m] = f32x4{0.f, 0.f, 0.f, 0.f};

  float best = -INFINITY;  // epilogue: running max over j of S * rq for row tid>>2
  const int er = tid >> 2;           // epilogue row
  const int eq = (tid & 3) * 4;      // epilogue first column of the quad
  const bool erow = tid < ROWS * 4;  // thread takes part in the epilogue

  const __amdgpu_buffer_rsrc_t qres = make_rsrc(query, uint32_t(Q) * C * 2);
  const int groups = (Q + COLS - 1) / COLS;
  for (int g = 0; g < groups; ++g) {
    const int qg0 = g * COLS;
    int qoff[NTG];
#pragma unroll
    for (int n = 0; n < NTG; ++n) {
      const int j = qg0 + n * 16 + row;
      qoff[n] = j < Q ? j * C * 2 : kOOB;
    }
    f32x4 S[MT][NTG];
    f32x4 QG[NTG];
#pragma unroll
    for (int n = 0; n < NTG; ++n) {
      QG[n] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int m = 0; m < MT; ++m) S[m][n] = f32x4{0.f, 0.f, 0.f, 0.f};
    }

    // Two register buffers of U channel steps each: the loads of the next
    // batch are in flight while the current batch feeds the MFMAs.  Only the
    // first query group also accumulates the Gram diagonal and the pooling.
    auto load_batch = [&](int ks0, bf16x8 (&a)[U][MT], bf16x8 (&b)[U][NTG]) {
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int ks = ks0 + u;
        const int c = ks * kKStep + grp * 8;
        const int cb = (ks < k_end && c < C) ? c * 2 : kOOB;
#pragma unroll
        for (int m = 0; m < MT; ++m) a[u][m] = buf_load_bf16x8(xres, xoff[m] + cb);
#pragma unroll
        for (int n = 0; n < NTG; ++n) b[u][n] = buf_load_bf16x8(qres, qoff[n] + cb);
      }
    };
    auto compute_batch = [&](int ks0, const bf16x8 (&a)[U][MT], const bf16x8 (&b)[U][NTG], auto pool) {
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int ks = ks0 + u;
#pragma unroll
        for (int n = 0; n < NTG; ++n) {
#pragma unroll
          for (int m = 0; m < MT; ++m)
            S[m][n] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[u][m], b[u][n], S[m][n], 0, 0, 0);
          QG[n] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(b[u][n], b[u][n], QG[n], 0, 0, 0);
        }
        if constexpr (decltype(pool)::value) {
          f32x4 P0 = {0.f, 0.f, 0.f, 0.f}, P1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int m = 0; m < MT; ++m) {
            G[m] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[u][m], a[u][m], G[m], 0, 0, 0);
            P0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[u][m], I0, P0, 0, 0, 0);
            P1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[u][m], I1, P1, 0, 0, 0);
          }
          float v0 = (P0[0] + P0[1]) + (P0[2] + P0[3]);
          float v1 = (P1[0] + P1[1]) + (P1[2] + P1[3]);
          v0 += __shfl_xor(v0, 16, kWave);
          v1 += __shfl_xor(v1, 16, kWave);
          v0 += __shfl_xor(v0, 32, kWave);
          v1 += __shfl_xor(v1, 32, kWave);
          // lanes 0-15 hold channels 32ks+0..15, lanes 16-31 channels 32ks+16..31;
          // a device-coherent store (the frame's last workgroup reads it back)
          const int ch = ks * kKStep + lane;
          const int off = (lane < 32 && ch < C && ks < k_end) ? ch * 4 : kOOB;
          __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(lane < 16 ? v0 : v1), pres, off, 0, kSc1);
        }
      }
    };
    auto stream_channels = [&](auto pool) {
      // sched_barrier keeps the compiler from sinking a prefetch next to its use
      bf16x8 a0[U][MT], b0[U][NTG], a1[U][MT], b1[U][NTG];
      load_batch(k_begin, a0, b0);
      for (int ks0 = k_begin; ks0 < k_end; ks0 += 2 * U) {
        load_batch(ks0 + U, a1, b1);
        __builtin_amdgcn_sched_barrier(0);
        compute_batch(ks0, a0, b0, pool);
        __builtin_amdgcn_sched_barrier(0);
        load_batch(ks0 + 2 * U, a0, b0);
        __builtin_amdgcn_sched_barrier(0);
        compute_batch(ks0 + U, a1, b1, pool);
        __builtin_amdgcn_sched_barrier(0);
      }
    };
    if (g == 0) stream_channels(std::true_type{});
    else stream_channels(std::false_type{});

    // ---- combine the waves' partial results (fixed order) ----
    const bool diag = (row >> 2) == grp;  // this lane holds a diagonal element
#pragma unroll
    for (int n = 0; n < NTG; ++n)
      if (diag) s_qpart[wave][n * 16 + row] = QG[n][row & 3];
    if (g == 0) {
#pragma unroll
      for (int m = 0; m < MT; ++m)
        if (diag) s_gpart[wave][m * 16 + row] = G[m][row & 3];
    }
    __syncthreads();
    if (tid < COLS && qg0 + tid < Q) {
      float s = 0.f;
#pragma unroll
      for (int w = 0; w < NW; ++w) s += s_qpart[w][tid];
      const float rq = s > 0.f ? 1.0f / sqrtf(s) : 0.f;
      s_rq[qg0 + tid] = rq;
      if (blockIdx.x == 0) rq_out[qg0 + tid] = rq;
    }
    if (g == 0 && tid < ROWS) {
      float s = 0.f;
#pragma unroll
      for (int w = 0; w < NW; ++w) s += s_gpart[w][tid];
      s_xn[tid] = sqrtf(s);
    }
    __syncthreads();
#pragma unroll
    for (int n = 0; n < NTG; ++n) {
#pragma unroll
      for (int m = 0; m < MT; ++m)
#pragma unroll
        for (int e = 0; e < 4; ++e) s_red[wave][m * 16 + 4 * grp + e][row] = S[m][n][e];
      __syncthreads();
      if (erow) {
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          float v = 0.f;
#pragma unroll
          for (int w = 0; w < NW; ++w) v += s_red[w][er][eq + k];
          const int j = qg0 + n * 16 + eq + k;
          if (j < Q && er < TM) best = fmaxf(best, v * s_rq[j]);
          s_red[0][er][eq + k] = v;
        }
      }
      __syncthreads();
      if (tid < 16) {
        const int j = qg0 + n * 16 + tid;
        if (j < Q) {
          float s = 0.f;
          for (int r = 0; r < TM; ++r) s += s_red[0][r][tid];
          st_dev(sig_part + part * Q + j, s);
        }
      }
      __syncthreads();
    }
  }

  if (erow) {
    best = fmaxf(best, __shfl_xor(best, 1, kWave));
    best = fmaxf(best, __shfl_xor(best, 2, kWave));
    if ((tid & 3) == 0 && er < TM) {
      const float xn = s_xn[er];
      tok_score[size_t(t) * N + tok0 + er] = xn > 0.f ? best / xn : 0.f;
    }
  }
  tile_finished(f, t, s_rq, s_dred, s_flag);
}

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
__global__ __launch_bounds__(kThreads) void k_relevance_valu(const In* __restrict__ X,
                                                             const In* __restrict__ query, int N,
                                                             int tile_tokens, float* __restrict__ tok_score,
                                                             float* __restrict__ rq_out, FrameArgs f) {
  constexpr int NW = kThreads / kWave;
  constexpr int V = Vec<In>::kN;
  constexpr int QB = 16;
  __shared__ float s_rq[kQMax];
  __shared__ float s_sig[NW][kQMax];
  __shared__ double s_dred[NW];
  __shared__ int s_flag[4];

  int t, tile;
  tile_of_block(blockIdx.x, f.tiles, t, tile);
  if (t >= f.T) return;
  const int C = f.C, Q = f.Q;
  const int tok0 = tile * tile_tokens;
  const int TM = min(tile_tokens, N - tok0);
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int nvec = C / V;
  const size_t part = size_t(t) * f.tiles + tile;
  float* pool_part = f.pool_part;
  float* sig_part = f.sig_part;

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
    if (lane == 0) {
      const float rq = s > 0.f ? 1.0f / sqrtf(s) : 0.f;
      s_rq[j] = rq;
      if (blockIdx.x == 0) rq_out[j] = rq;
    }
  }
  for (int j = tid; j < NW * kQMax; j += kThreads) (&s_sig[0][0])[j] = 0.f;
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
      tok_score[size_t(t) * N + tok0 + r] = xn > 0.f ? best / xn : 0.f;
    }
  }

  // channel sums of the tile (tokens in order)
  for (int v = tid; v < nvec; v += kThreads) {
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
    for (int i = 0; i < V; ++i) st_dev(pool_part + part * C + v * V + i, acc[i]);
  }
  __syncthreads();
  for (int j = tid; j < Q; j += kThreads) {
    float s = 0.f;
    for (int w = 0; w < NW; ++w) s += s_sig[w][j];
    st_dev(sig_part + part * Q + j, s);
  }
  tile_finished(f, t, s_rq, s_dred, s_flag);
}

#ifndef WZ_REL_U
#define WZ_REL_U 2  // channel steps per register buffer (two buffers in flight)
#endif

template <int MT, int NTG>
void launch_mfma_variant(const wz_config& c, const Tiling& tl, const void* X, const void* query,
                         float* tok_score, float* rq, const FrameArgs& fa, hipStream_t s) {
  constexpr int U = NTG <= 2 ? WZ_REL_U : 2;
  hipLaunchKernelGGL((k_relevance_mfma<MT, NTG, U>), dim3(tl.grid), dim3(kThreads), 0, s,
                     static_cast<const uint16_t*>(X), static_cast<const uint16_t*>(query), c.H * c.W,
                     tl.tile_tokens, tok_score, rq, fa);
}

template <int MT>
void launch_mfma_mt(const wz_config& c, const Tiling& tl, const void* X, const void* query, float* tok_score,
                    float* rq, const FrameArgs& fa, hipStream_t s) {
  const int nt = (c.Q + 15) / 16;
  if (nt <= 1) launch_mfma_variant<MT, 1>(c, tl, X, query, tok_score, rq, fa, s);
  else if (nt <= 2) launch_mfma_variant<MT, 2>(c, tl, X, query, tok_score, rq, fa, s);
  else launch_mfma_variant<MT, 4>(c, tl, X, query, tok_score, rq, fa, s);
}

}  // namespace

bool relevance_uses_mfma(const wz_config& c) { return c.in_dtype == WZ_BF16 && c.Q >= 16; }

hipError_t launch_relevance(const wz_config& c, const void* X, const void* query, float* tok_score,
                            float* frame_rel, float* frame_delta, const Workspace& ws, hipStream_t s) {
  const Tiling tl = relevance_tiling(c);
  FrameArgs fa{ws.pool_part, ws.sig_part, ws.pooled, ws.pnorm2, ws.ctr, frame_rel, frame_delta,
               c.T, c.C, c.Q, tl.tiles_per_frame};
  if (relevance_uses_mfma(c)) {
    if (tl.mtiles == 1) launch_mfma_mt<1>(c, tl, X, query, tok_score, ws.rq, fa, s);
    else launch_mfma_mt<2>(c, tl, X, query, tok_score, ws.rq, fa, s);
  } else if (c.in_dtype == WZ_BF16) {
    hipLaunchKernelGGL((k_relevance_valu<uint16_t>), dim3(tl.grid), dim3(kThreads), 0, s,
                       static_cast<const uint16_t*>(X), static_cast<const uint16_t*>(query), c.H * c.W,
                       tl.tile_tokens, tok_score, ws.rq, fa);
  } else {
    hipLaunchKernelGGL((k_relevance_valu<float>), dim3(tl.grid), dim3(kThreads), 0, s,
                       static_cast<const float*>(X), static_cast<const float*>(query), c.H * c.W,
                       tl.tile_tokens, tok_score, ws.rq, fa);
  }
  return hipGetLastError();
}

}  // namespace wz
