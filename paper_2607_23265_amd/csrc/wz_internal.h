// Internal declarations shared by the gfx950 kernels and the C-ABI layer.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "wavezip.h"

namespace wz {

constexpr int kWave = 64;

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// bf16 <-> fp32 (bf16 is the upper half of an fp32 bit pattern).
__device__ __forceinline__ float bf16_lo(uint32_t v) { return __uint_as_float(v << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t v) { return __uint_as_float(v & 0xffff0000u); }
__device__ __forceinline__ uint32_t f32_to_bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return 0x7fc0u;  // NaN stays NaN
  return (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
}

// Butterfly sum across the 64 lanes of a wave (every lane gets the total).
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, kWave);
  return v;
}
__device__ __forceinline__ double wave_sum_f64(double v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, kWave);
  return v;
}

// ---------------------------------------------------------------------------
// Tiling of the relevance pass: every workgroup owns one tile of up to 32
// consecutive tokens of one frame and reads all C channels of them.
// ---------------------------------------------------------------------------
constexpr int kXcds = 8;  // MI355X: workgroups are dealt to the 8 XCDs round robin

struct Tiling {
  int tiles_per_frame;  // ceil(N / tile_tokens)
  int tile_tokens;      // tokens per tile (the last tile of a frame may be shorter)
  int mtiles;           // 16-row MFMA tiles per workgroup tile
  int grid;             // workgroups: frames rounded up to a multiple of kXcds, times tiles
};

inline Tiling relevance_tiling(const wz_config& c) {
  const int N = c.H * c.W;
  const int cap = 32;  // two 16-row MFMA tiles
  Tiling t;
  t.tiles_per_frame = (N + cap - 1) / cap;
  t.tile_tokens = (N + t.tiles_per_frame - 1) / t.tiles_per_frame;
  t.mtiles = (t.tile_tokens + 15) / 16;
  t.grid = (c.T + kXcds - 1) / kXcds * kXcds * t.tiles_per_frame;
  return t;
}

// Workgroup b handles frame t = (b / kXcds / tiles) * kXcds + b % kXcds and
// tile (b / kXcds) % tiles, so every tile of a frame runs on the same XCD
// (its L2 then holds the partial sums the frame's last workgroup combines).
__device__ __forceinline__ void tile_of_block(int b, int tiles, int& t, int& tile) {
  const int xcd = b % kXcds, slot = b / kXcds;
  tile = slot % tiles;
  t = (slot / tiles) * kXcds + xcd;
}

// Counters the relevance pass uses to find the last workgroup of a frame and
// of a pair of adjacent frames.  They sit at the start of the workspace, are
// left at zero by every call, and must be zero before the first call.
constexpr int kMaxFrames = 2048;
struct Counters {
  int frame[kMaxFrames];     // tiles of frame t finished
  int pair[kMaxFrames + 1];  // frames t-1, t finished (for delta_t)
};

// Workspace carve-up (all offsets 256-byte aligned).
struct Workspace {
  Counters* ctr;       // zero between calls
  float* pool_part;    // [T][tiles][C]  per-tile channel sums
  float* sig_part;     // [T][tiles][Q]  per-tile sums of x . q_j
  float* pooled;       // [T][C]         per-frame channel sums p_t
  double* pnorm2;      // [T]            |p_t|^2
  float* rq;           // [Q]            1 / |q_j| (0 for a zero query token)
  float* tok_score;    // [T*N]
  float* frame_rel;    // [T]
  float* frame_delta;  // [T]
  int32_t* budget;     // [T]
  int32_t* offset;     // [T+1]
  size_t bytes;
};

inline size_t align256(size_t v) { return (v + 255) & ~size_t(255); }

inline Workspace workspace_layout(const wz_config& c, char* base) {
  const Tiling tl = relevance_tiling(c);
  const size_t T = c.T, N = size_t(c.H) * c.W, C = c.C, Q = c.Q, tiles = tl.tiles_per_frame;
  Workspace w;
  size_t off = 0;
  auto take = [&](size_t bytes) { char* p = base ? base + off : nullptr; off += align256(bytes); return p; };
  w.ctr = reinterpret_cast<Counters*>(take(sizeof(Counters)));
  w.pool_part = reinterpret_cast<float*>(take(T * tiles * C * 4));
  w.sig_part = reinterpret_cast<float*>(take(T * tiles * Q * 4));
  w.pooled = reinterpret_cast<float*>(take(T * C * 4));
  w.pnorm2 = reinterpret_cast<double*>(take(T * 8));
  w.rq = reinterpret_cast<float*>(take(Q * 4));
  w.tok_score = reinterpret_cast<float*>(take(T * N * 4));
  w.frame_rel = reinterpret_cast<float*>(take(T * 4));
  w.frame_delta = reinterpret_cast<float*>(take(T * 4));
  w.budget = reinterpret_cast<int32_t*>(take(T * 4));
  w.offset = reinterpret_cast<int32_t*>(take((T + 1) * 4));
  w.bytes = off;
  return w;
}

// Kernel launchers (each returns hipGetLastError() of its launches).
hipError_t launch_relevance(const wz_config& c, const void* X, const void* query, float* tok_score,
                            float* frame_rel, float* frame_delta, const Workspace& ws, hipStream_t s);
hipError_t launch_temporal_budget(const wz_config& c, const float* frame_rel, const float* frame_delta,
                                  int32_t* budget, int32_t* offset, float* rel_rect, hipStream_t s);
hipError_t launch_spatial_condense(const wz_config& c, const void* X, const float* tok_score,
                                   const int32_t* budget, const int32_t* offset, void* out_tokens,
                                   int32_t* out_index, hipStream_t s);

}  // namespace wz
