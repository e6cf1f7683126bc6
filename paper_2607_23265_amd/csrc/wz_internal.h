// Internal declarations shared by the gfx950 kernels and the C-ABI layer.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>

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
// Decomposition of the relevance pass (shapes and limits; the kernels'
// comments give the details).  Token-tiled path: tiles of at most 64 tokens
// with every channel.  MFMA-layout path: a token tile of a frame (up to 256
// tokens) and one slice of channels; tiles cover whole frames when H*W <= 256,
// so the query, which every workgroup must read for its channels, is read
// about once per frame, and channel slices give the grid enough workgroups.
// Vector-ALU path: tiles of up to 32 tokens, all channels.
// ---------------------------------------------------------------------------
constexpr int kXcds = 8;          // MI355X: workgroups are dealt to the 8 XCDs round robin
constexpr int kCUs = 256;
constexpr int kMaxWaves = 16;     // 16-row MFMA tiles per token tile
constexpr int kTilesPerWave = 2;  // 16-row MFMA tiles per wave on the MFMA path
constexpr int kSliceSteps = 32;   // 32-channel steps per slice at most (the query slice sits in LDS)
constexpr int kTokMax = 4096;     // validated bound on tokens per frame

// Query columns of the per-slice partial scores, padded for 16-byte rows.
inline int qpad(int Q) { return (Q + 3) & ~3; }

// Streaming kernels of the relevance pass, chosen by shape:
//   kRelTok  bf16, Q <= 64 or 128 < Q <= 256: token tiles with every
//            channel, each wave a channel stripe with its own LDS-transposed
//            MFMA (above 64 query tokens, passes of 32 columns per tile);
//   kRelWg   bf16, 64 < Q <= 128: token tiles with every channel, the
//            workgroup's waves sharing each channel chunk of the tile and the
//            query in LDS, each wave some 16-row tiles against every column;
//   kRelMfma bf16, Q > 256, frames of >= 49 tokens: MFMA-layout loads;
//   kRelValu everything else (fp32 inputs, small frames with many queries).
enum RelKind { kRelValu = 0, kRelMfma = 1, kRelTok = 2, kRelWg = 3 };
RelKind relevance_kind(const wz_config& c);

struct RelPlan {
  RelKind kind;
  int tiles;        // token tiles per frame
  int tile_tokens;  // tokens per tile (the last tile of a frame may be shorter)
  int mt;           // 16-row MFMA tiles per token tile (kRelMfma)
  int slices;       // channel slices
  int kc;           // channels per slice
  int grid;         // workgroups: frames rounded up to a multiple of kXcds, x tiles x slices
  int threads;      // threads per workgroup
  int ipc;          // kRelTok: row load instructions per chunk (tile rows / 8)
  int ntg;          // kRelTok, kRelWg: 16-column query tiles
  int rtw;          // kRelWg: 16-row tiles per wave (tiles of up to 64 * rtw tokens)
};

inline RelPlan relevance_plan(const wz_config& c) {
  const int N = c.H * c.W;
  RelPlan p{};
  p.kind = relevance_kind(c);
  if (p.kind == kRelTok) {
    // tiles of 16 to 64 tokens with every channel, one slice.  A workgroup
    // fills a CU's LDS, so a CU runs (workgroups / CUs rounded up) of them one
    // after another, each loading its tile's tokens and the query's 16-row
    // tiles: take the tile count with the fewest rows loaded per CU, the
    // smaller count on a tie
    const int tr = (c.T + kXcds - 1) / kXcds * kXcds;
    // query tiles: 1, 2 or 4 of 16 columns; above 64 columns, passes of 32
    const int nq = c.Q <= 16 ? 16 : c.Q <= 32 ? 32 : c.Q <= 64 ? 64 : 32;
    const int lo = (N + 63) / 64, hi = std::max(lo, (N + 15) / 16);
    long best = -1;
    for (int k = lo; k <= hi; ++k) {
      const int rows = (N + k - 1) / k + nq;
      const long cost = long((long(tr) * k + kCUs - 1) / kCUs) * rows;
      if (best < 0 || cost < best) best = cost, p.tiles = k;
    }
    p.tile_tokens = (N + p.tiles - 1) / p.tiles;
    p.ipc = (p.tile_tokens + 7) / 8;
    p.ntg = nq / 16;
    p.mt = 0;
    p.slices = 1;
    p.kc = c.C;
    p.threads = 8 * 64;  // (the launcher takes four waves for one pass of two query tiles)
  } else if (p.kind == kRelWg) {
    // tiles of at most 128 tokens; two workgroups share a CU.  Every
    // workgroup streams its tile's rows and the whole query through LDS:
    // take the tile count with the fewest rows streamed per CU slot, the
    // smaller count on a tie
    const int tr = (c.T + kXcds - 1) / kXcds * kXcds;
    p.ntg = c.Q <= 16 ? 1 : c.Q <= 32 ? 2 : c.Q <= 64 ? 4 : 8;
    const int lo = (N + 127) / 128, hi = std::max(lo, (N + 15) / 16);
    long best = -1;
    for (int k = lo; k <= hi; ++k) {
      const int rows = (N + k - 1) / k + 16 * p.ntg;
      const long cost = long((long(tr) * k + 2 * kCUs - 1) / (2 * kCUs)) * rows;
      if (best < 0 || cost < best) best = cost, p.tiles = k;
    }
    p.tile_tokens = (N + p.tiles - 1) / p.tiles;
    p.rtw = p.tile_tokens <= 64 ? 1 : 2;
    p.mt = 0;
    p.slices = 1;
    p.kc = c.C;
    p.threads = 256;
  } else if (p.kind == kRelMfma) {
    const int cap = 16 * kMaxWaves;
    p.tiles = (N + cap - 1) / cap;
    p.tile_tokens = (N + p.tiles - 1) / p.tiles;
    p.mt = (p.tile_tokens + 15) / 16;
    const int ksteps = (c.C + 31) / 32;
    // slices of at most kSliceSteps steps; more while the grid is short of
    // one workgroup per CU, keeping slices of at least 8 channel steps and
    // per-slice partial scores (4*Q bytes a token) under a quarter of X (2*C)
    const int smin = (ksteps + kSliceSteps - 1) / kSliceSteps;
    const int smax = std::max(smin, std::min(ksteps / 8, c.C / (8 * c.Q)));
    int S = smin;
    while (S < smax && (long long)c.T * p.tiles * S < kCUs) ++S;
    const int kper = (ksteps + S - 1) / S;
    p.kc = kper * 32;
    p.slices = (ksteps + kper - 1) / kper;
    p.threads = (p.mt + kTilesPerWave - 1) / kTilesPerWave * 64;
  } else {
    const int cap = 32;
    p.tiles = (N + cap - 1) / cap;
    p.tile_tokens = (N + p.tiles - 1) / p.tiles;
    p.mt = (p.tile_tokens + 15) / 16;
    p.slices = 1;
    p.kc = c.C;
    p.threads = 256;
  }
  p.grid = (c.T + kXcds - 1) / kXcds * kXcds * p.tiles * p.slices;
  return p;
}

// Workgroup b works on frame t = (b / kXcds / (tiles*slices)) * kXcds + b % kXcds,
// so every workgroup of a frame runs on the same XCD.
__device__ __forceinline__ void unit_of_block(int b, int tiles, int slices, int& t, int& tile, int& slice) {
  const int xcd = b % kXcds, slot = b / kXcds;
  const int per_frame = tiles * slices;
  const int r = slot % per_frame;
  t = (slot / per_frame) * kXcds + xcd;
  tile = r / slices;
  slice = r % slices;
}

constexpr int kMaxFrames = 2048;
// frames up to which the budget is folded into the selection kernel (one
// wave computes it: up to 64 frames in registers, up to 256 four frames per
// lane in LDS); above, one workgroup of its own computes it once, which costs
// less than every selection workgroup repeating a workgroup-wide budget
constexpr int kFusedTMax = 256;

// Workspace carve-up (all offsets 256-byte aligned).
// Bytes of the filter-bank operator rows in the workspace (0 if unused).
size_t filter_rows_bytes(const wz_config& c);

struct Workspace {
  float* s_part;       // [T][slices][N][qpad(Q)] per-slice x . q_j (only with several slices)
  float* g_part;       // [T][slices][N]          per-slice |x|^2 (only with several slices)
  float* qg_part;      // [T][slices][Q]          per-slice |q_j|^2
  float* sig_part;     // [T][tiles][slices][Q]   per-unit sums over tokens of x . q_j
  float* pool_part;    // [T][tiles][C]           per-tile channel sums
  float* tok_score;    // [T*N]
  int32_t* rank;       // [T*N]                   selection rank of each token in its frame
  int32_t* byrank;     // [T*N]                   token of each rank
  float* gate;         // [T*N]                   saliency gate of each token's 2x2 block
  float* gate2;        // [T*N]                   level-2 gate of each token (two spatial levels)
  float* frame_rel;    // [T]
  float* frame_delta;  // [T]
  int32_t* budget;     // [T]
  int32_t* offset;     // [T+1]
  uint16_t* frows;     // [B][2][pad(H*W)]        filter-bank operator rows (bf16 inputs, filter spatial basis)
  size_t bytes;
};

inline size_t align256(size_t v) { return (v + 255) & ~size_t(255); }

// split: room for the filter-bank operator rows when the problem uses them
// (without it the modulator runs its fused form, which keeps them in LDS).
inline Workspace workspace_layout(const wz_config& c, char* base, bool split = true) {
  const RelPlan pl = relevance_plan(c);
  const size_t T = c.T, N = size_t(c.H) * c.W, C = c.C, Q = c.Q, QP = qpad(c.Q), tiles = pl.tiles,
               S = pl.slices;
  Workspace w;
  size_t off = 0;
  auto take = [&](size_t bytes) { char* p = base ? base + off : nullptr; off += align256(bytes); return p; };
  w.s_part = reinterpret_cast<float*>(take(S > 1 ? T * S * N * QP * 4 : 0));
  w.g_part = reinterpret_cast<float*>(take(S > 1 ? T * S * N * 4 : 0));
  w.qg_part = reinterpret_cast<float*>(take(T * S * Q * 4));
  w.sig_part = reinterpret_cast<float*>(take(T * tiles * S * Q * 4));
  w.pool_part = reinterpret_cast<float*>(take(T * tiles * C * 4));
  w.tok_score = reinterpret_cast<float*>(take(T * N * 4));
  w.rank = reinterpret_cast<int32_t*>(take(T * N * 4));
  w.byrank = reinterpret_cast<int32_t*>(take(T * N * 4));
  w.gate = reinterpret_cast<float*>(take(T * N * 4));
  w.gate2 = reinterpret_cast<float*>(take(c.spatial_levels == 2 ? T * N * 4 : 0));
  w.frame_rel = reinterpret_cast<float*>(take(T * 4));
  w.frame_delta = reinterpret_cast<float*>(take(T * 4));
  w.budget = reinterpret_cast<int32_t*>(take(T * 4));
  w.offset = reinterpret_cast<int32_t*>(take((T + 1) * 4));
  const size_t frows = split ? filter_rows_bytes(c) : 0;
  w.frows = frows ? reinterpret_cast<uint16_t*>(take(frows)) : nullptr;
  w.bytes = off;
  return w;
}

// Several videos in one launch: video v = blockIdx.y of every kernel works
// on X + v*x, query + v*q, the workspace and every intermediate kept in it
// + v*ws, out_tokens + v*out, out_index + v*idx, budget + v*bud and
// offset + v*off (byte strides).  Each kernel receives one argument set per
// video, so its body sees a single video.
constexpr int kMaxVideos = 8;
struct Videos {
  int V = 1;
  long long x = 0, q = 0, ws = 0, out = 0, idx = 0, bud = 0, off = 0;
  // the V problems are V queries over one video (x = 0): when shared_pass
  // holds they share one pass over X, and problem v > 0 reads the channel
  // sums of problem 0's workspace
  bool shared_x = false;
};
// queries of one video that one token-tiled pass serves together (its 64
// query columns at most); passes over X share them when this is 2 or more
inline int queries_per_pass(const wz_config& c) { return relevance_kind(c) == kRelTok ? 64 / c.Q : 1; }
inline bool shared_pass(const wz_config& c, int V) { return V > 1 && queries_per_pass(c) >= 2; }
template <typename A>
struct VideoArgs {
  A v[kMaxVideos];
};
template <typename P>
__host__ __device__ inline P* advance(P* p, long long bytes) {
  return p ? reinterpret_cast<P*>(reinterpret_cast<uintptr_t>(p) + bytes) : p;
}
inline Workspace advance(const Workspace& w, long long bytes) {
  Workspace o = w;
  o.s_part = advance(w.s_part, bytes);
  o.g_part = advance(w.g_part, bytes);
  o.qg_part = advance(w.qg_part, bytes);
  o.sig_part = advance(w.sig_part, bytes);
  o.pool_part = advance(w.pool_part, bytes);
  o.tok_score = advance(w.tok_score, bytes);
  o.rank = advance(w.rank, bytes);
  o.byrank = advance(w.byrank, bytes);
  o.gate = advance(w.gate, bytes);
  o.gate2 = advance(w.gate2, bytes);
  o.frame_rel = advance(w.frame_rel, bytes);
  o.frame_delta = advance(w.frame_delta, bytes);
  o.budget = advance(w.budget, bytes);
  o.offset = advance(w.offset, bytes);
  o.frows = advance(w.frows, bytes);
  return o;
}

// Kernel launchers (each returns hipGetLastError() of its launches; `vs`
// batches videos, one by default).
// Streaming pass of stage 1: per-unit partials into ws (and a_{t,n} into
// tok_score when there is one channel slice).
hipError_t launch_relevance_stream(const wz_config& c, const void* X, const void* query, float* tok_score,
                                   const Workspace& ws, hipStream_t s, const Videos& vs = Videos{});
// Per-frame finish of stage 1: a_{t,n} (several slices), r_t and delta_t;
// with `order` also every frame's selection ranks and block gates (into
// ws.rank, ws.byrank, ws.gate) for launch_assign_gather.
hipError_t launch_frame(const wz_config& c, const Workspace& ws, float* tok_score, float* frame_rel,
                        float* frame_delta, bool order, hipStream_t s, const Videos& vs = Videos{});
// Budgets alone, in one workgroup (wz_temporal_budget, and wz_condense when
// T > kFusedTMax).
hipError_t launch_budget(const wz_config& c, const float* frame_rel, const float* frame_delta, int32_t* budget,
                         int32_t* offset, float* rel_rect, hipStream_t s, const Videos& vs = Videos{});
// Selection, spatial modulation and compaction.  With offset_in the frames'
// row offsets are given; without it (T <= kFusedTMax) every workgroup computes
// the budgets from frame_rel and frame_delta itself and workgroup 0 writes
// them to budget_out / offset_out when those are not null.  With ws the
// frames' ranks and gates come from launch_frame; without it each workgroup
// forms its frame's from tok_score.
hipError_t launch_assign_gather(const wz_config& c, const void* X, const float* tok_score, const float* frame_rel,
                                const float* frame_delta, const int32_t* offset_in, const Workspace* ws,
                                int32_t* budget_out, int32_t* offset_out, void* out_tokens, int32_t* out_index,
                                hipStream_t s, const Videos& vs = Videos{});
// Workgroups per frame of launch_assign_gather for V videos at once.
int assign_groups_per_frame(const wz_config& c, int V = 1);
// Selection, spatial modulation with the db4 / bior4.4 filter bank of
// c.spatial_basis, and compaction, from the scores and the frames' row
// offsets (each workgroup ranks its frame itself).  Needs
// filter_assign_supported(c).
bool filter_assign_supported(const wz_config& c);
// With rank (the per-frame kernel's selection ranks, [T][H*W]) each workgroup
// reads its frame's ranks instead of forming them.  With rows (bf16 inputs; at
// least filter_rows_bytes(c) bytes, 16-byte aligned) the split form runs: a
// row kernel forms each kept token's operator row once per frame into rows,
// then a contraction kernel applies them to the frame's channels; without it
// one fused kernel per (frame, channel slice) forms the rows it uses.
// Whether the filter-bank modulator computes the budgets itself (T <= 64,
// Haar temporal basis, and LDS for them without fewer rows per chunk).
bool filter_budget_folds(const wz_config& c);
// With fb.rel set (filter_budget_folds(c), rank given; offset unused)
// the kernel computes the budgets itself from fb.rel and fb.delta ([T] r_t
// and delta_t) and writes them to fb.budget ([T], may be null) and the row
// offsets to fb.offset ([T+1]).
struct FoldedBudget {
  const float* rel = nullptr;
  const float* delta = nullptr;
  int32_t* budget = nullptr;
  int32_t* offset = nullptr;
};
hipError_t launch_filter_assign(const wz_config& c, const void* X, const float* tok_score, const int32_t* offset,
                                const int32_t* rank, uint16_t* rows, void* out_tokens, int32_t* out_index,
                                hipStream_t s, const Videos& vs = Videos{}, const FoldedBudget& fb = FoldedBudget{});

}  // namespace wz
