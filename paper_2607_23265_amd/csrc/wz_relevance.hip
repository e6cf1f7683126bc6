// Stage 1, streaming part: the similarity-branch Cross-Modal Scorer (Sec.
// 3.2.1) and the pooled features of the Visual Change Estimator (Sec. 3.2.2,
// Eq. (8)) in ONE kernel that reads the frames once.  Per token it needs
//     x . q_j  (all j),  |x|^2,  |q_j|^2,
// and per frame the channel sums p_t = sum_n x_{t,n} (the mean's cosine is the
// sum's) and sigma_j = sum_n x_{t,n} . q_j = p_t . q_j.  It writes them per
// work unit; the per-frame kernel adds the units' partials in a fixed order
// and forms r_t and delta_t (and a_{t,n} when a unit holds only some channels).
//
// Three decompositions, chosen by shape:
//  * token tiles (bf16, Q <= 64; below): a workgroup owns up to 64 tokens of a
//    frame with every channel, so a_{t,n} is final in the pass;
//  * MFMA layout (bf16, Q > 64, frames of >= 49 tokens): a workgroup owns one
//    token tile of one frame (the whole frame when H*W <= 256; each wave holds
//    two 16-row MFMA tiles) and one slice of at most 32 x 32 channels.  It
//    stages the slice of the query (MFMA B layout) in LDS, where every wave
//    reads it; X streams into A-operand registers through an R-deep ring of
//    16-byte buffer loads with no barrier in the loop.  Per 32-channel step
//    each wave runs v_mfma_f32_16x16x32_bf16 for
//        S += X Q^T      (the relevance contraction),
//        G += X X^T      (diagonal: |x|^2),
//        P += X I        (identity columns: channel sums of its tokens),
//    and one wave per step adds the query's Gram matrix (diagonal: |q_j|^2).
//    With one slice the workgroup also finishes its tokens' a_{t,n}; with
//    several it writes the partial x . q_j and |x|^2;
//  * vector ALU (fp32 inputs, small frames with many queries): tiles of up to
//    32 tokens over all channels, one wave per token, wave-reduced dot
//    products.
#include <type_traits>

#include "wz_device.h"

namespace wz {
namespace {

constexpr int kKStep = 32;    // channels per MFMA K step (16x16x32)
constexpr int kQMax = 1024;   // validated bound on query tokens

// Per-unit outputs of the streaming pass (layouts in the workspace carve-up).
struct StreamArgs {
  const void* X;      // [T][H][W][C]
  const void* query;  // [Q][C]
  float* s_part;
  float* g_part;
  float* qg_part;
  float* sig_part;
  float* pool_part;
  float* tok_score;  // written here when there is one slice
  int T, N, C, Q, QP, tiles, slices;
  // several queries in one pass (token-tiled path): `query` holds groups x qg
  // rows (Q = groups * qg); query g's scores, column sums and norms go to the
  // buffers above advanced by g * gws bytes, its channel sums are query 0's
  int groups = 1, qg = 0;
  long long gws = 0;
};
static_assert(sizeof(VideoArgs<StreamArgs>) <= 4096, "per-video arguments exceed the kernel argument limit");

// ---------------------------------------------------------------------------
// MFMA path
// ---------------------------------------------------------------------------
// NTG: 16-column query tiles per pass over the slice (queries of more tokens
// take several passes); R: depth of the X prefetch ring in 32-channel steps.
template <int NTG, int R>
__global__ __launch_bounds__(kMaxWaves / kTilesPerWave * 64) void k_relevance_mfma(
    int tile_tokens, int kc, const VideoArgs<StreamArgs> va) {
  const StreamArgs f = va.v[blockIdx.y];
  const uint16_t* __restrict__ X = static_cast<const uint16_t*>(f.X);
  const uint16_t* __restrict__ query = static_cast<const uint16_t*>(f.query);
  constexpr int MTW = kTilesPerWave;
  constexpr int MAXW = kMaxWaves / MTW;
  constexpr int QB = 8;                          // query units staged per thread per batch
  __shared__ u32x4 s_q[kSliceSteps][NTG][kWave];  // the group's query slice, MFMA B layout
  __shared__ float s_poolw[MAXW][kSliceSteps * kKStep];  // per-wave channel sums of the slice
  __shared__ float s_colw[MAXW][NTG * 16];       // per-wave column sums of S
  __shared__ float s_qgw[MAXW][NTG * 16];        // per-wave |q_j|^2 partials
  __shared__ float s_xt[kMaxWaves * 16];         // |x| of the tile's tokens (one slice)
  __shared__ float s_rq[kQMax];                 // 1/|q_j| (one slice)

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
        v0 = row_sum4(v0);
        v1 = row_sum4(v1);
        // lanes 0-15: channels 32ks+0..15 of the slice, lanes 16-31: 32ks+16..31
        if (lane < 32) s_poolw[wave][ks * kKStep + lane] = lane < 16 ? v0 : v1;
      }
    };
    // Steps 2s and 2s+1 read the two 64-byte halves of the same 128-byte
    // line of each row, so they are consumed and re-issued as a pair: the
    // second request of a line then finds the first one's miss in flight
    // instead of a line the cache may have evicted meanwhile.
    static_assert(R % 2 == 0, "the ring advances in pairs of steps");
    auto run = [&](auto pool) {
      for (int ks0 = 0; ks0 < kper; ks0 += R) {
#pragma unroll
        for (int r = 0; r < R; r += 2) {
          const int ks = ks0 + r;
          if (ks < kper) compute(ks, a[r], pool);
          if (ks + 1 < kper) compute(ks + 1, a[r + 1], pool);
          issue(ks + R, a[r]);
          issue(ks + 1 + R, a[r + 1]);
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
      v = row_sum4(v);
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
          else buf_store_f32(gg, gres, r < TM ? (tok0 + r) * 4 : kOOB);
        }
      }
      // the slice's channel sums, waves added in order
      const __amdgpu_buffer_rsrc_t pres =
          make_rsrc(f.pool_part + (size_t(t) * f.tiles + tile) * C, uint32_t(C) * 4);
      for (int c = tid; c < kper * kKStep; c += nthreads) {
        float s = 0.f;
        for (int w = 0; w < nw; ++w) s += s_poolw[w][c];
        buf_store_f32(s, pres, c_lo + c < c_hi ? (c_lo + c) * 4 : kOOB);
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
        if (S == 1) s_rq[j] = qq > 0.f ? 1.0f / sqrtf(qq) : 0.f;
        if (tile == 0) f.qg_part[(size_t(t) * S + sl) * Q + j] = qq;
        f.sig_part[((size_t(t) * f.tiles + tile) * S + sl) * Q + j] = sg;
      }
    }
    __syncthreads();
    const __amdgpu_buffer_rsrc_t sres =
        make_rsrc(f.s_part + (size_t(t) * S + sl) * N * QP, S > 1 ? uint32_t(N) * QP * 4 : 0u);
#pragma unroll
    for (int n = 0; n < NTG; ++n) {
      const int j = qg0 + n * 16 + row;  // this lane's column
      if (S == 1) {
        const float rq = j < Q ? s_rq[j] : 0.f;
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
            buf_store_f32(Sacc[i][n][e], sres, (r < TM && j < Q) ? ((tok0 + r) * QP + j) * 4 : kOOB);
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
}

// bf16 dot2 helpers of the token-tiled path
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ float dot2(uint32_t a, uint32_t b, float c) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, a), __builtin_bit_cast(bf16x2, b), c, false);
}
// Selector pairs for channel sums: dot2(x, (1, 0)) picks the low bf16 of x,
// dot2(x, (0, 1)) the high one.  They must reach the instruction in VGPRs:
// this compiler encodes the pair (1, 0) as the inline constant 1.0, which the
// hardware reads as (0, 1) for a packed bf16 operand.
constexpr uint32_t kBf16OneLo = 0x00003F80u;  // bf16 pair (1, 0)
constexpr uint32_t kBf16OneHi = 0x3F800000u;  // bf16 pair (0, 1)

// ---------------------------------------------------------------------------
// Token-tiled path (bf16, Q <= 64)
// ---------------------------------------------------------------------------
// A workgroup owns one tile of at most 64 tokens of one frame with ALL its
// channels, so a_{t,n} is final here and no per-slice partial scores are
// written; its tokens are one contiguous stretch of X.  The W waves (eight;
// four for one pass of two query tiles with the channel sums in LDS, where
// that measured faster) split the channels into 64-channel chunks (wave w
// takes chunks w, w + W, ...) and never wait for each other until the
// epilogue.  Per chunk a wave
//   1. loads the tile's rows and the query's rows for the chunk (8 rows x 128
//      bytes per instruction, whole cache lines; the query is L2-resident);
//   2. stores both to its own LDS buffers (16-byte units XOR-swizzled by row)
//      and, from the same registers, accumulates |x|^2, |q_j|^2 and the
//      chunk's channel sums with bf16 dot2 instructions; the channel sums are
//      reduced across the wave by DPP and lane swaps and gathered in LDS;
//   3. runs two 32-channel steps of S += X Q^T (v_mfma_f32_16x16x32_bf16) on
//      four 16-row tiles, reading both operands from its buffers;
//   4. re-issues the ring slot for the chunk after next.
// In the epilogue each wave first reduces its own accumulator rows to
// sigma_j (lane swaps); then the waves' partial S, |x|^2, |q_j|^2 and sigma_j
// are added in wave order through LDS (two barriers), a_{t,n} = max_j S_nj /
// (|q_j| |x_n|) is formed, and the tile's channel sums leave in one coalesced
// store.
constexpr int kTokWaves = 8;
constexpr int kTokChunk = 64;      // channels per chunk (128 bytes of a bf16 row)
constexpr int kTokRows = 64;       // tokens per tile at most (four 16-row MFMA tiles)
constexpr int kTokPoolMax = 8192;  // channels whose sums are gathered in LDS
constexpr int kTokQMax = 256;      // query tokens: at most four passes of 64 over a tile

// POOL: the tile's channel sums are gathered in LDS (C <= kTokPoolMax) and
// stored once at the end; otherwise a few lanes store them chunk by chunk.
// MODE kTokOne: one pass over the tile for every query column;
// kTokGroups: the query columns are f.groups queries of f.qg tokens each,
// a_{t,n} taken per query; kTokPasses: queries of more than NQ tokens, one
// pass over the tile per NQ query rows (its later reads mostly from cache),
// a_{t,n} the maximum over the passes, the channel sums taken in the first.
enum TokMode { kTokOne = 0, kTokGroups = 1, kTokPasses = 2 };
// WV: the workgroup's waves.
template <int NTG, int IPC, bool POOL, int MODE, int WV = kTokWaves>
__global__ __launch_bounds__(WV * 64) void k_relevance_tok(int tile_tokens, const VideoArgs<StreamArgs> va) {
  constexpr int kTokRowsPerThread = kTokRows * 8 / (WV * kWave);  // epilogue rows of a thread (8 threads a row)
  static_assert(kTokRowsPerThread * WV * kWave == kTokRows * 8, "whole epilogue rows per thread");
  const StreamArgs f = va.v[blockIdx.y];
  const uint16_t* __restrict__ X = static_cast<const uint16_t*>(f.X);
  const uint16_t* __restrict__ query = static_cast<const uint16_t*>(f.query);
  constexpr int NQ = NTG * 16;  // query rows of the accumulators
  constexpr int QI = NQ / 8;    // query load instructions per chunk
  // chunks of loads in flight per wave: two (eight waves keep 16 chunks of
  // the tile in flight; deeper rings measured slower)
  constexpr int D = 2;
  // per-wave chunk buffers (16-byte units swizzled by row): rows 0 .. 63 of a
  // wave's region stage its tile rows, rows 64 .. 64 + NQ - 1 its query rows;
  // after the loop the region holds the wave's partial S [64 rows][NQ] floats
  __shared__ __align__(16) u32x4 s_xq[WV][kTokRows + NQ][8];
  __shared__ __align__(16) float s_pool[POOL ? kTokPoolMax : 4];
  __shared__ float s_xx[WV][kTokRows];
  __shared__ float s_qq[WV][NQ];
  __shared__ float s_rq[NQ];
  __shared__ float s_sig[WV][NQ];  // per-wave column sums of S

  int t, tile, sl;
  unit_of_block(blockIdx.x, f.tiles, 1, t, tile, sl);
  if (t >= f.T) return;
  const int N = f.N, C = f.C, Q = f.Q;
  const int tok0 = tile * tile_tokens;
  const int TM = min(tile_tokens, N - tok0);
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int r16 = lane & 15, grp = lane >> 4;  // MFMA layout: row / column, K group
  const int lr = lane >> 3, lu = lane & 7;     // load layout: row lr of each 8-row group, 16-byte unit lu
  const int nch = (C + kTokChunk - 1) / kTokChunk;

  const __amdgpu_buffer_rsrc_t xres = make_rsrc_uniform(X + (size_t(t) * N + tok0) * C, uint32_t(TM) * C * 2);
  constexpr bool GR = MODE == kTokGroups;
  const int npass = MODE == kTokPasses ? (Q + NQ - 1) / NQ : 1;
  float best_all[kTokRowsPerThread];
#pragma unroll
  for (int k = 0; k < kTokRowsPerThread; ++k) best_all[k] = -INFINITY;
  for (int h = 0; h < npass; ++h) {
    const int qb = h * NQ, Qh = min(NQ, Q - qb);
    const bool sums = h == 0;
    const __amdgpu_buffer_rsrc_t qres = make_rsrc_uniform(query + size_t(qb) * C, uint32_t(Qh) * C * 2);

    // ring slot: the tile's rows 8k + lr and the query's rows 8k + lr, unit lu
    // of the chunk; chunks past the end, rows past the tile or the query and
    // channels past C read zeros
    struct Slot {
      bf16x8 x[IPC];
      bf16x8 q[QI];
    };
    // (query rows past Qh lie past the end of qres and read zeros; a per-lane
    // row test here would become a branch around the load)
    auto issue = [&](int c, Slot& d) {
      const int cc = c * kTokChunk + 8 * lu;
      const bool ok = c < nch && cc < C;
#pragma unroll
      for (int k = 0; k < IPC; ++k) d.x[k] = buf_load_bf16x8(xres, ok ? (8 * k + lr) * C * 2 + cc * 2 : kOOB);
#pragma unroll
      for (int k = 0; k < QI; ++k) d.q[k] = buf_load_bf16x8(qres, ok ? (8 * k + lr) * C * 2 + cc * 2 : kOOB);
    };

    f32x4 Sacc[4][NTG];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int n = 0; n < NTG; ++n) Sacc[i][n] = f32x4{0.f, 0.f, 0.f, 0.f};
    float xx[IPC], qq[QI];
#pragma unroll
    for (int k = 0; k < IPC; ++k) xx[k] = 0.f;
#pragma unroll
    for (int k = 0; k < QI; ++k) qq[k] = 0.f;
    uint32_t one_lo = kBf16OneLo, one_hi = kBf16OneHi;
    asm volatile("" : "+v"(one_lo), "+v"(one_hi));  // opaque: keeps them out of inline constants
    float* pool = POOL ? s_pool : f.pool_part + (size_t(t) * f.tiles + tile) * C;

    auto consume = [&](int c, const Slot& d) {
      // rows to LDS; |x|^2, |q_j|^2 and channel sums from the registers
      float cs[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) cs[e] = 0.f;
#pragma unroll
      for (int k = 0; k < IPC; ++k) {
        const int row = 8 * k + lr;
        const u32x4 v = __builtin_bit_cast(u32x4, d.x[k]);
        s_xq[wave][row][lu ^ (row & 7)] = v;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          xx[k] = dot2(v[e], v[e], xx[k]);
          cs[2 * e] = dot2(v[e], one_lo, cs[2 * e]);
          cs[2 * e + 1] = dot2(v[e], one_hi, cs[2 * e + 1]);
        }
      }
#pragma unroll
      for (int k = 0; k < QI; ++k) {
        const int row = 8 * k + lr;
        const u32x4 v = __builtin_bit_cast(u32x4, d.q[k]);
        s_xq[wave][kTokRows + row][lu ^ (row & 7)] = v;
#pragma unroll
        for (int e = 0; e < 4; ++e) qq[k] = dot2(v[e], v[e], qq[k]);
      }
      // channel sums over the wave's rows (lanes lu, lu + 8, ..., lu + 56, in a
      // fixed order): lane 8 lr + lu ends with channel 8 lu + lr's
      const float cw = lane_transpose_sum8(cs);
      const int c0 = c * kTokChunk + 8 * lu;
      if (sums && c0 < C) pool[c0 + lr] = cw;
    };
    auto contract = [&]() {
#pragma unroll
      for (int st = 0; st < 2; ++st) {
        bf16x8 A[4], B[NTG];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int row = 16 * i + r16;
          A[i] = __builtin_bit_cast(bf16x8, s_xq[wave][row][(4 * st + grp) ^ (row & 7)]);
        }
#pragma unroll
        for (int n = 0; n < NTG; ++n) {
          const int row = 16 * n + r16;
          B[n] = __builtin_bit_cast(bf16x8, s_xq[wave][kTokRows + row][(4 * st + grp) ^ (row & 7)]);
        }
#pragma unroll
        for (int n = 0; n < NTG; ++n)
#pragma unroll
          for (int i = 0; i < 4; ++i)
            Sacc[i][n] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A[i], B[n], Sacc[i][n], 0, 0, 0);
      }
    };

    // rows this wave never loads (8 * IPC .. 63) are zero in its buffer
    for (int u = 8 * IPC * 8 + lane; u < kTokRows * 8; u += kWave) (&s_xq[wave][0][0])[u] = u32x4{0u, 0u, 0u, 0u};

    // A ring of D slots: the wave's chunks c, c + 8, ..., c + 8 (D - 1) are in
    // flight while it works on the oldest.  The loads are issued in slot
    // order before and in the loop, and the norms' updates are pinned before
    // a slot's reload: otherwise the slot needs a second register set and a
    // copy at the end of the loop, and the compiler waits for the whole ring
    // once per iteration.
    auto pin = [&]() {
#pragma unroll
      for (int k = 0; k < IPC; ++k) asm volatile("" : "+v"(xx[k]));
#pragma unroll
      for (int k = 0; k < QI; ++k) asm volatile("" : "+v"(qq[k]));
    };
    Slot ring[D];
#pragma unroll
    for (int s = 0; s < D; ++s) {
      issue(wave + s * WV, ring[s]);
      __builtin_amdgcn_sched_barrier(0);
    }
    for (int c0 = wave; c0 < nch; c0 += D * WV) {
#pragma unroll
      for (int s = 0; s < D; ++s) {
        const int c = c0 + s * WV;
        __builtin_amdgcn_sched_barrier(0);
        if (c < nch) {
          consume(c, ring[s]);
          pin();
          contract();
        }
        issue(c + D * WV, ring[s]);
      }
    }

    // ---- epilogue: waves added in order; LDS-only barriers, so nothing waits
    // for outstanding global accesses ----
    auto row8_sum = [](float v) {  // the 8 lanes of a load-layout row
      v += __uint_as_float(__builtin_amdgcn_update_dpp(0u, __float_as_uint(v), 0xB1, 0xF, 0xF, false));   // lane ^ 1
      v += __uint_as_float(__builtin_amdgcn_update_dpp(0u, __float_as_uint(v), 0x4E, 0xF, 0xF, false));   // lane ^ 2
      v += __uint_as_float(__builtin_amdgcn_update_dpp(0u, __float_as_uint(v), 0x141, 0xF, 0xF, false));  // 7 - i in 8
      return v;
    };
#pragma unroll
    for (int k = 0; k < IPC; ++k) {
      const float v = row8_sum(xx[k]);
      if (lu == 0) s_xx[wave][8 * k + lr] = v;
    }
    for (int r = 8 * IPC + lane; r < kTokRows; r += kWave) s_xx[wave][r] = 0.f;
#pragma unroll
    for (int k = 0; k < QI; ++k) {
      const float v = row8_sum(qq[k]);
      if (lu == 0) s_qq[wave][8 * k + lr] = v;
    }
    // sigma_j of the wave: its accumulator column j = 16 n + r16 summed over the
    // wave's 64 rows (rows past the tile hold zeros), the four lane groups by
    // lane swaps
#pragma unroll
    for (int n = 0; n < NTG; ++n) {
      float v = 0.f;
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int e = 0; e < 4; ++e) v += Sacc[i][n][e];
      const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
      v = __uint_as_float(a[0]) + __uint_as_float(a[1]);
      const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
      v = __uint_as_float(b[0]) + __uint_as_float(b[1]);
      if (lane < 16) s_sig[wave][16 * n + r16] = v;
    }
    // wave w's partial S sits in its own region: [row][NQ] floats from &s_xq[w][0][0]
    static_assert((kTokRows + NQ) * 8 * 16 >= kTokRows * NQ * 4, "partial S fits the wave's region");
    auto s_part = [&](int w, int r, int j) -> float& { return reinterpret_cast<float*>(&s_xq[w][0][0])[r * NQ + j]; };
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int n = 0; n < NTG; ++n)
#pragma unroll
        for (int e = 0; e < 4; ++e) s_part(wave, 16 * i + 4 * grp + e, 16 * n + r16) = Sacc[i][n][e];
    lds_barrier();  // every sum below reads the waves' partials in wave order
    if (tid < Qh) {
      float v = 0.f, qv = 0.f;
#pragma unroll
      for (int w = 0; w < WV; ++w) {
        v += s_sig[w][tid];
        qv += s_qq[w][tid];
      }
      if constexpr (GR) {
        const int g = tid / f.qg, j = tid - g * f.qg;
        advance(f.sig_part, g * f.gws)[(size_t(t) * f.tiles + tile) * f.qg + j] = v;
        if (tile == 0) advance(f.qg_part, g * f.gws)[size_t(t) * f.qg + j] = qv;
      } else {
        f.sig_part[(size_t(t) * f.tiles + tile) * Q + qb + tid] = v;
        if (tile == 0) f.qg_part[size_t(t) * Q + qb + tid] = qv;
      }
    }
    if (tid < NQ) {
      float qv = 0.f;
      for (int w = 0; w < WV; ++w) qv += s_qq[w][tid];
      s_rq[tid] = qv > 0.f ? 1.0f / sqrtf(qv) : 0.f;
    }
    // thread -> rows tid / 8 + RS k (k < kTokRowsPerThread), columns CPT * (tid % 8) .. + CPT - 1;
    // every row's partials are read before the first barrier (the query maxima below reuse wave 0's region)
    constexpr int CPT = NQ / 8;
    constexpr int RS = WV * kWave / 8;  // rows the threads cover at once
    const int cg = (tid & 7) * CPT;
    float sv[kTokRowsPerThread][CPT], x2[kTokRowsPerThread];
#pragma unroll
    for (int k = 0; k < kTokRowsPerThread; ++k) {
      const int row = (tid >> 3) + RS * k;
#pragma unroll
      for (int e = 0; e < CPT; ++e) {
        float v = 0.f;
#pragma unroll
        for (int w = 0; w < WV; ++w) v += s_part(w, row, cg + e);
        sv[k][e] = v;
      }
      x2[k] = 0.f;
#pragma unroll
      for (int w = 0; w < WV; ++w) x2[k] += s_xx[w][row];
    }
    lds_barrier();  // 1 / |q_j| in s_rq
    float rq[CPT];
#pragma unroll
    for (int e = 0; e < CPT; ++e) rq[e] = s_rq[cg + e];
    if constexpr (GR) {
      // the rows' S_nj / |q_j| into LDS (wave 0's region: every read of the
      // partials is behind the last barrier); thread g of a row's eight takes
      // the maximum over query g's columns
      float* s_cos = reinterpret_cast<float*>(&s_xq[0][0][0]);  // [64 rows][NQ]
#pragma unroll
      for (int k = 0; k < kTokRowsPerThread; ++k)
#pragma unroll
        for (int e = 0; e < CPT; ++e) s_cos[((tid >> 3) + RS * k) * NQ + cg + e] = sv[k][e] * rq[e];
      lds_barrier();
      const int g = tid & 7;
#pragma unroll
      for (int k = 0; k < kTokRowsPerThread; ++k) {
        const int row = (tid >> 3) + RS * k;
        if (g < f.groups && row < TM) {
          float best = -INFINITY;
          for (int j = 0; j < f.qg; ++j) best = fmaxf(best, s_cos[row * NQ + g * f.qg + j]);
          const float xn = sqrtf(x2[k]);
          advance(f.tok_score, g * f.gws)[size_t(t) * N + tok0 + row] = xn > 0.f ? best / xn : 0.f;
        }
      }
    } else {
#pragma unroll
      for (int k = 0; k < kTokRowsPerThread; ++k) {
        const int row = (tid >> 3) + RS * k;
        float best = -INFINITY;
#pragma unroll
        for (int e = 0; e < CPT; ++e)
          if (cg + e < Qh) best = fmaxf(best, sv[k][e] * rq[e]);
        best = fmaxf(best, __uint_as_float(__builtin_amdgcn_update_dpp(0u, __float_as_uint(best), 0xB1, 0xF, 0xF, false)));
        best = fmaxf(best, __uint_as_float(__builtin_amdgcn_update_dpp(0u, __float_as_uint(best), 0x4E, 0xF, 0xF, false)));
        best = fmaxf(best, __uint_as_float(__builtin_amdgcn_update_dpp(0u, __float_as_uint(best), 0x141, 0xF, 0xF, false)));
        best_all[k] = fmaxf(best_all[k], best);
        if (h == npass - 1 && (tid & 7) == 0 && row < TM) {
          const float xn = sqrtf(x2[k]);
          f.tok_score[size_t(t) * N + tok0 + row] = xn > 0.f ? best_all[k] / xn : 0.f;
        }
      }
    }
    if (h + 1 < npass) lds_barrier();  // the next pass rewrites every wave's region
  }

  if (POOL) {
    const __amdgpu_buffer_rsrc_t pres =
        make_rsrc_uniform(f.pool_part + (size_t(t) * f.tiles + tile) * C, uint32_t(C) * 4);
    for (int c4 = tid; c4 < C / 4; c4 += WV * kWave)
      buf_store_wt_b128(reinterpret_cast<const u32x4*>(s_pool)[c4], pres, c4 * 16);
  }
}

// ---------------------------------------------------------------------------
// Workgroup-shared token tiles (bf16, 64 < Q <= 128)
// ---------------------------------------------------------------------------
// With a wide query, per-wave channel stripes (above) would stage the query
// once per wave and add every wave's partial S through LDS.  Here the eight
// waves of a workgroup share each 64-channel chunk: the tile's rows (up to
// 64 * RTW tokens) and the query's 128 rows are loaded once per workgroup
// (one 16-byte unit per thread and row group, whole cache lines), staged in a
// double-buffered LDS stage (16-byte units XOR-swizzled by row), and the
// waves tile S as 2 row groups x 4 column groups: wave (wr, wc) contracts
// 16-row tiles wr * 2 RTW .. wr * 2 RTW + 2 RTW - 1 against 16-column tiles
// 2 wc, 2 wc + 1.  |x|^2, |q_j|^2 and the chunk's channel sums come from the
// load registers (bf16 dot2), the channel sums added over the waves in wave
// order through LDS.  One LDS-only barrier per chunk; D chunks of loads in
// flight in registers.  The row maxima and column sums of S are combined
// across the waves through LDS at the end, in a fixed order.  Two
// workgroups share a CU.
constexpr int kWgQMax = 128;  // query tokens of the workgroup-shared path
constexpr int kWgWaves = 8;
constexpr int kWgNQ = 128;    // query rows the stage holds (eight 16-column tiles)

template <int RTW>
__global__ __launch_bounds__(kWgWaves * 64, 2) void k_relevance_wg(int tile_tokens, const VideoArgs<StreamArgs> va) {
  const StreamArgs f = va.v[blockIdx.y];
  constexpr int RT = 64 * RTW;                 // tile rows the stage holds
  constexpr int NQ = kWgNQ;
  constexpr int MTW = 2 * RTW;                 // 16-row tiles per wave
  constexpr int NTW = 2;                       // 16-column tiles per wave
  constexpr int XR = RT / 64;                  // tile rows each thread loads per chunk
  constexpr int QR = NQ / 64;                  // query rows each thread loads per chunk
  constexpr int D = 2 + (RTW == 1);            // chunks of loads in flight
  __shared__ __align__(16) u32x4 s_x[2][RT][8];
  __shared__ __align__(16) u32x4 s_q[2][NQ][8];
  __shared__ __align__(16) float s_pp[2][kWgWaves][kTokChunk];  // per-wave channel sums of a chunk
  __shared__ float s_xx[RT];
  __shared__ float s_qq[NQ];
  __shared__ float s_sig[2][NQ];    // column sums of S per row group
  __shared__ float s_best[4][RT];   // row maxima of S_nj / |q_j| per column group

  int t, tile, sl;
  unit_of_block(blockIdx.x, f.tiles, 1, t, tile, sl);
  if (t >= f.T) return;
  const uint16_t* __restrict__ X = static_cast<const uint16_t*>(f.X);
  const uint16_t* __restrict__ query = static_cast<const uint16_t*>(f.query);
  const int N = f.N, C = f.C, Q = f.Q;
  const int tok0 = tile * tile_tokens;
  const int TM = min(tile_tokens, N - tok0);
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wr = wave >> 2, wc = wave & 3;     // row group, column group
  const int r16 = lane & 15, grp = lane >> 4;  // MFMA layout: row / column, K group
  const int rb = tid >> 3, lu = tid & 7;       // load layout: rows rb + 64 k, 16-byte unit lu
  const int nch = (C + kTokChunk - 1) / kTokChunk;

  const __amdgpu_buffer_rsrc_t xres = make_rsrc_uniform(X + (size_t(t) * N + tok0) * C, uint32_t(TM) * C * 2);
  const __amdgpu_buffer_rsrc_t qres = make_rsrc_uniform(query, uint32_t(Q) * C * 2);
  const __amdgpu_buffer_rsrc_t pres =
      make_rsrc_uniform(f.pool_part + (size_t(t) * f.tiles + tile) * C, uint32_t(C) * 4);

  struct Slot {
    bf16x8 x[XR];
    bf16x8 q[QR];
  };
  // chunk c's units; chunks past the end, rows past the tile or the query
  // and channels past C read zeros (query rows past Q <= NQ lie past the end
  // of qres; a per-lane row test here would become a branch around the load)
  auto issue = [&](int c, Slot& d) {
    const int cc = c * kTokChunk + 8 * lu;
    const bool ok = c < nch && cc < C;
#pragma unroll
    for (int k = 0; k < XR; ++k) d.x[k] = buf_load_bf16x8(xres, ok ? (rb + 64 * k) * C * 2 + cc * 2 : kOOB);
#pragma unroll
    for (int k = 0; k < QR; ++k) d.q[k] = buf_load_bf16x8(qres, ok ? (rb + 64 * k) * C * 2 + cc * 2 : kOOB);
  };

  f32x4 Sacc[MTW][NTW];
#pragma unroll
  for (int i = 0; i < MTW; ++i)
#pragma unroll
    for (int n = 0; n < NTW; ++n) Sacc[i][n] = f32x4{0.f, 0.f, 0.f, 0.f};
  float xx[XR], qq[QR];
#pragma unroll
  for (int k = 0; k < XR; ++k) xx[k] = 0.f;
#pragma unroll
  for (int k = 0; k < QR; ++k) qq[k] = 0.f;
  uint32_t one_lo = kBf16OneLo, one_hi = kBf16OneHi;
  asm volatile("" : "+v"(one_lo), "+v"(one_hi));  // opaque: keeps them out of inline constants

  // units to the chunk's stage; norms and channel sums from the registers
  auto consume = [&](int c, const Slot& d) {
    const int b = c & 1;
    float cs[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) cs[e] = 0.f;
#pragma unroll
    for (int k = 0; k < XR; ++k) {
      const int row = rb + 64 * k;
      const u32x4 v = __builtin_bit_cast(u32x4, d.x[k]);
      s_x[b][row][lu ^ (row & 7)] = v;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        xx[k] = dot2(v[e], v[e], xx[k]);
        cs[2 * e] = dot2(v[e], one_lo, cs[2 * e]);
        cs[2 * e + 1] = dot2(v[e], one_hi, cs[2 * e + 1]);
      }
    }
#pragma unroll
    for (int k = 0; k < QR; ++k) {
      const int row = rb + 64 * k;
      const u32x4 v = __builtin_bit_cast(u32x4, d.q[k]);
      s_q[b][row][lu ^ (row & 7)] = v;
#pragma unroll
      for (int e = 0; e < 4; ++e) qq[k] = dot2(v[e], v[e], qq[k]);
    }
    // the wave's channel sums (lanes lu, lu + 8, ..., lu + 56, in a fixed
    // order): lane 8 k + lu ends with channel 8 lu + k's
    s_pp[b][wave][8 * lu + (lane >> 3)] = lane_transpose_sum8(cs);
  };
  // chunk c's channel sums, the waves' added in wave order by wave 0 (lane k:
  // channel k of the chunk).  Every lane of every wave issues the store (all
  // but wave 0's past the end of the buffer, which drops them), so the count of
  // memory operations in flight is the same on every path and the waits for
  // the ring's loads stay exact; the sums themselves sit behind a scalar branch.
  auto pool_out = [&](int c) {
    const int b = c & 1;
    float v = 0.f;
    if (wave == 0) {
#pragma unroll
      for (int w = 0; w < kWgWaves; ++w) v += s_pp[b][w][lane];
    }
    const int ch = c * kTokChunk + lane;
    __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v), pres, (wave == 0 && ch < C) ? ch * 4 : kOOB, 0,
                                          kWriteThrough);
  };
  auto contract = [&](int c) {
    const int b = c & 1;
#pragma unroll
    for (int st = 0; st < 2; ++st) {
      bf16x8 B[NTW];
#pragma unroll
      for (int n = 0; n < NTW; ++n) {
        const int row = 16 * (NTW * wc + n) + r16;
        B[n] = __builtin_bit_cast(bf16x8, s_q[b][row][(4 * st + grp) ^ (row & 7)]);
      }
#pragma unroll
      for (int i = 0; i < MTW; ++i) {
        const int rt = MTW * wr + i;
        if (16 * rt < TM) {
          const int row = 16 * rt + r16;
          const bf16x8 A = __builtin_bit_cast(bf16x8, s_x[b][row][(4 * st + grp) ^ (row & 7)]);
#pragma unroll
          for (int n = 0; n < NTW; ++n) Sacc[i][n] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A, B[n], Sacc[i][n], 0, 0, 0);
        }
      }
    }
  };

  // The loop runs to a multiple of D chunks: a chunk past the end reads
  // zeros, adds nothing and stores nowhere, and no branch around a load or
  // store makes the compiler wait for the whole ring.  The loads are issued
  // in slot order before and in the loop (the waits count the loads issued
  // after a slot's), and the norms' updates may not sink below a slot's
  // reload: the slot would need a second register set, and the copy back at
  // the end of the loop waits for the whole ring.
  Slot ring[D];
#pragma unroll
  for (int s = 0; s < D; ++s) {
    issue(s, ring[s]);
    __builtin_amdgcn_sched_barrier(0);
  }
  for (int c0 = 0; c0 < nch; c0 += D) {
#pragma unroll
    for (int s = 0; s < D; ++s) {
      const int c = c0 + s;
      __builtin_amdgcn_sched_barrier(0);
      consume(c, ring[s]);
#pragma unroll
      for (int k = 0; k < XR; ++k) asm volatile("" : "+v"(xx[k]));
#pragma unroll
      for (int k = 0; k < QR; ++k) asm volatile("" : "+v"(qq[k]));
      lds_barrier();  // chunk c staged by every wave; chunk c - 2's stage no longer read
      issue(c + D, ring[s]);
      pool_out(c);
      contract(c);
    }
  }

  // ---- epilogue ----
  auto row8_sum = [](float v) {  // the 8 lanes of a load-layout row
    v += __uint_as_float(__builtin_amdgcn_update_dpp(0u, __float_as_uint(v), 0xB1, 0xF, 0xF, false));   // lane ^ 1
    v += __uint_as_float(__builtin_amdgcn_update_dpp(0u, __float_as_uint(v), 0x4E, 0xF, 0xF, false));   // lane ^ 2
    v += __uint_as_float(__builtin_amdgcn_update_dpp(0u, __float_as_uint(v), 0x141, 0xF, 0xF, false));  // 7 - i in 8
    return v;
  };
#pragma unroll
  for (int k = 0; k < XR; ++k) {
    const float v = row8_sum(xx[k]);
    if (lu == 0) s_xx[rb + 64 * k] = v;
  }
#pragma unroll
  for (int k = 0; k < QR; ++k) {
    const float v = row8_sum(qq[k]);
    if (lu == 0) s_qq[rb + 64 * k] = v;
  }
  // sigma_j of the wave's rows: accumulator column j = 16 n + r16, the four
  // lane groups added by lane swaps (rows past the tile hold zeros)
#pragma unroll
  for (int n = 0; n < NTW; ++n) {
    float v = 0.f;
#pragma unroll
    for (int i = 0; i < MTW; ++i)
#pragma unroll
      for (int e = 0; e < 4; ++e) v += Sacc[i][n][e];
    v = row_sum4(v);
    if (lane < 16) s_sig[wr][16 * (NTW * wc + n) + r16] = v;
  }
  lds_barrier();  // s_qq, s_xx, s_sig complete
  if (tid < Q) {
    f.sig_part[(size_t(t) * f.tiles + tile) * Q + tid] = s_sig[0][tid] + s_sig[1][tid];
    if (tile == 0) f.qg_part[size_t(t) * Q + tid] = s_qq[tid];
  }
  // the wave's row maxima of S_nj / |q_j| over its columns j < Q
  float rq[NTW];
  bool live[NTW];
#pragma unroll
  for (int n = 0; n < NTW; ++n) {
    const int j = 16 * (NTW * wc + n) + r16;
    const float qv = s_qq[j];
    rq[n] = qv > 0.f ? 1.0f / sqrtf(qv) : 0.f;
    live[n] = j < Q;
  }
#pragma unroll
  for (int i = 0; i < MTW; ++i) {
    const int rt = MTW * wr + i;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      float best = -INFINITY;
#pragma unroll
      for (int n = 0; n < NTW; ++n)
        if (live[n]) best = fmaxf(best, Sacc[i][n][e] * rq[n]);
      best = fmaxf(best, __uint_as_float(__builtin_amdgcn_update_dpp(0u, __float_as_uint(best), 0xB1, 0xF, 0xF, false)));
      best = fmaxf(best, __uint_as_float(__builtin_amdgcn_update_dpp(0u, __float_as_uint(best), 0x4E, 0xF, 0xF, false)));
      best = fmaxf(best, __uint_as_float(__builtin_amdgcn_update_dpp(0u, __float_as_uint(best), 0x141, 0xF, 0xF, false)));
      best = fmaxf(best, __uint_as_float(__builtin_amdgcn_update_dpp(0u, __float_as_uint(best), 0x140, 0xF, 0xF, false)));
      if (r16 == e) s_best[wc][16 * rt + 4 * grp + e] = best;
    }
  }
  lds_barrier();  // s_best complete
  // a_{t,n} = max_j S_nj / (|q_j| |x_n|): the column groups' maxima in order
  for (int row = tid; row < TM; row += kWgWaves * 64) {
    const float best = fmaxf(fmaxf(s_best[0][row], s_best[1][row]), fmaxf(s_best[2][row], s_best[3][row]));
    const float xn = sqrtf(s_xx[row]);
    f.tok_score[size_t(t) * N + tok0 + row] = xn > 0.f ? best / xn : 0.f;
  }
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
__global__ __launch_bounds__(256) void k_relevance_valu(int tile_tokens, const VideoArgs<StreamArgs> va) {
  const StreamArgs f = va.v[blockIdx.y];
  const In* __restrict__ X = static_cast<const In*>(f.X);
  const In* __restrict__ query = static_cast<const In*>(f.query);
  constexpr int NW = 4;
  constexpr int V = Vec<In>::kN;
  constexpr int QB = 16;
  __shared__ float s_rq[kQMax];
  __shared__ float s_sig[NW][kQMax];

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
    if (lane == 0) {
      s_rq[j] = s > 0.f ? 1.0f / sqrtf(s) : 0.f;
      if (tile == 0) f.qg_part[size_t(t) * Q + j] = s;
    }
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

  // channel sums of the tile (tokens in order)
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
    for (int i = 0; i < V; ++i) f.pool_part[part * C + v * V + i] = acc[i];
  }
  __syncthreads();
  for (int j = tid; j < Q; j += 256) {
    float s = 0.f;
    for (int w = 0; w < NW; ++w) s += s_sig[w][j];
    f.sig_part[part * Q + j] = s;
  }
}

#ifndef WZ_REL_RING
#define WZ_REL_RING 4  // X prefetch depth in 32-channel steps (MFMA-layout path)
#endif

template <int NTG>
void launch_mfma(const RelPlan& pl, const VideoArgs<StreamArgs>& va, int V, hipStream_t s) {
  hipLaunchKernelGGL((k_relevance_mfma<NTG, WZ_REL_RING>), dim3(pl.grid, V), dim3(pl.threads), 0, s, pl.tile_tokens,
                     pl.kc, va);
}

template <int NTG, int IPC, int MODE>
void launch_tok_mode(const RelPlan& pl, const VideoArgs<StreamArgs>& va, int V, hipStream_t s) {
  const int C = va.v[0].C;
  // Four waves for a query of 17 to 32 tokens in one pass with the channel
  // sums in LDS (measured faster than eight).  A pass shared by queries of
  // that size (64 query columns) takes four waves too: a wave's chunks set
  // the order in which each query's sums are added, so that each query's
  // results are bitwise those of its own pass.
  const bool four = MODE == kTokGroups ? (va.v[0].qg + 15) / 16 == 2 && C <= kTokPoolMax
                                       : NTG == 2 && MODE == kTokOne && C <= kTokPoolMax;
  // with 64 query columns the staging regions leave no room for the gathered channel sums
  if constexpr (NTG <= 2) {
    if (C <= kTokPoolMax) {
      if constexpr (NTG == 2 && MODE == kTokOne) {
        if (four) {
          hipLaunchKernelGGL((k_relevance_tok<NTG, IPC, true, MODE, 4>), dim3(pl.grid, V), dim3(4 * kWave), 0, s,
                             pl.tile_tokens, va);
          return;
        }
      }
      hipLaunchKernelGGL((k_relevance_tok<NTG, IPC, true, MODE>), dim3(pl.grid, V), dim3(kTokWaves * kWave), 0, s,
                         pl.tile_tokens, va);
      return;
    }
  }
  if constexpr (NTG == 4 && MODE == kTokGroups) {
    if (four) {
      hipLaunchKernelGGL((k_relevance_tok<NTG, IPC, false, MODE, 4>), dim3(pl.grid, V), dim3(4 * kWave), 0, s,
                         pl.tile_tokens, va);
      return;
    }
  }
  hipLaunchKernelGGL((k_relevance_tok<NTG, IPC, false, MODE>), dim3(pl.grid, V), dim3(kTokWaves * kWave), 0, s,
                     pl.tile_tokens, va);
}
template <int NTG, int IPC>
void launch_tok(const RelPlan& pl, const VideoArgs<StreamArgs>& va, int V, hipStream_t s) {
  if (va.v[0].groups > 1) {
    launch_tok_mode<NTG, IPC, kTokGroups>(pl, va, V, s);
  } else if (va.v[0].Q > 16 * NTG) {
    // the plan takes two query tiles for passes (checked by the caller)
    if constexpr (NTG == 2) launch_tok_mode<NTG, IPC, kTokPasses>(pl, va, V, s);
  } else {
    launch_tok_mode<NTG, IPC, kTokOne>(pl, va, V, s);
  }
}

}  // namespace

RelKind relevance_kind(const wz_config& c) {
  if (c.in_dtype != WZ_BF16) return kRelValu;
  if (c.Q > 64 && c.Q <= kWgQMax) return kRelWg;
  if (c.Q <= kTokQMax) return kRelTok;
  // two 16-row MFMA tiles per wave, at least 2 waves: frames of at least 49 tokens
  return c.H * c.W >= 49 ? kRelMfma : kRelValu;
}

hipError_t launch_relevance_stream(const wz_config& c, const void* X, const void* query, float* tok_score,
                                   const Workspace& ws, hipStream_t s, const Videos& vs) {
  RelPlan pl = relevance_plan(c);
  VideoArgs<StreamArgs> va{};
  int V = vs.V;
  if (vs.shared_x && shared_pass(c, vs.V)) {
    // queries in groups of up to 64 columns, one pass over X per group (grid
    // y = group): the per-query plan's tiles, query tiles for a group's columns
    const int G = std::min(vs.V, queries_per_pass(c));
    const int QT = c.Q * G;
    pl.ntg = QT <= 16 ? 1 : QT <= 32 ? 2 : 4;
    V = (vs.V + G - 1) / G;
    for (int e = 0; e < V; ++e) {
      const int q0 = e * G, n = std::min(G, vs.V - q0);
      const Workspace w = advance(ws, q0 * vs.ws);
      va.v[e] = StreamArgs{X, advance(query, q0 * vs.q), w.s_part, w.g_part, w.qg_part, w.sig_part, w.pool_part,
                           advance(tok_score, q0 * vs.ws), c.T, c.H * c.W, c.C, c.Q * n, qpad(c.Q * n), pl.tiles,
                           pl.slices, n, c.Q, vs.ws};
    }
  } else {
    for (int v = 0; v < vs.V; ++v) {
      const Workspace w = advance(ws, v * vs.ws);
      va.v[v] = StreamArgs{advance(X, v * vs.x), advance(query, v * vs.q), w.s_part, w.g_part, w.qg_part,
                           w.sig_part, w.pool_part, advance(tok_score, v * vs.ws), c.T, c.H * c.W, c.C, c.Q,
                           qpad(c.Q), pl.tiles, pl.slices};
    }
  }
  if (pl.kind == kRelTok) {
    // columns beyond the query tiles are served by passes of two tiles only
    if (va.v[0].Q > 16 * pl.ntg && (pl.ntg != 2 || va.v[0].groups > 1)) return hipErrorInvalidValue;
#define WZ_TOK(NTG)                                 \
  switch (pl.ipc) {                                 \
    case 1: launch_tok<NTG, 1>(pl, va, V, s); break; \
    case 2: launch_tok<NTG, 2>(pl, va, V, s); break; \
    case 3: launch_tok<NTG, 3>(pl, va, V, s); break; \
    case 4: launch_tok<NTG, 4>(pl, va, V, s); break; \
    case 5: launch_tok<NTG, 5>(pl, va, V, s); break; \
    case 6: launch_tok<NTG, 6>(pl, va, V, s); break; \
    case 7: launch_tok<NTG, 7>(pl, va, V, s); break; \
    default: launch_tok<NTG, 8>(pl, va, V, s); break; \
  }
    if (pl.ntg == 1) { WZ_TOK(1) } else if (pl.ntg == 2) { WZ_TOK(2) } else { WZ_TOK(4) }
#undef WZ_TOK
  } else if (pl.kind == kRelWg) {
    if (va.v[0].groups > 1 || va.v[0].Q > kWgNQ) return hipErrorInvalidValue;
    if (pl.rtw == 1)
      hipLaunchKernelGGL((k_relevance_wg<1>), dim3(pl.grid, V), dim3(kWgWaves * 64), 0, s, pl.tile_tokens, va);
    else
      hipLaunchKernelGGL((k_relevance_wg<2>), dim3(pl.grid, V), dim3(kWgWaves * 64), 0, s, pl.tile_tokens, va);
  } else if (pl.kind == kRelMfma) {
    // queries of more than 32 tokens take several passes of 32 over the slice:
    // wider query groups no longer fit the accumulators in registers
    launch_mfma<2>(pl, va, V, s);
  } else if (c.in_dtype == WZ_BF16) {
    hipLaunchKernelGGL((k_relevance_valu<uint16_t>), dim3(pl.grid, V), dim3(pl.threads), 0, s, pl.tile_tokens, va);
  } else {
    hipLaunchKernelGGL((k_relevance_valu<float>), dim3(pl.grid, V), dim3(pl.threads), 0, s, pl.tile_tokens, va);
  }
  return hipGetLastError();
}

}  // namespace wz
