// Stage 1, streaming part: the similarity-branch Cross-Modal Scorer (Sec.
// 3.2.1) and the pooled features of the Visual Change Estimator (Sec. 3.2.2,
// Eq. (8)) in ONE kernel that reads the frames once.  Per token it needs
//     x . q_j  (all j),  |x|^2,  |q_j|^2,
// and per frame the channel sums p_t = sum_n x_{t,n} (the mean's cosine is the
// sum's) and sigma_j = sum_n x_{t,n} . q_j = p_t . q_j.  It writes them per
// work unit; the frame kernel adds the units' partials in a fixed order and
// forms a_{t,n}, r_t and delta_t.
//
// Work decomposition (MFMA path: bf16 inputs, Q >= 16, frames of >= 49 tokens).
// A workgroup owns one token tile of one frame (the whole frame when
// H*W <= 256; each wave holds two 16-row MFMA tiles) and one slice of at most
// 32 x 32 channels.  At the start it stages the slice of the query (MFMA B
// layout) in LDS, where every wave reads it; X streams from HBM into A-operand
// registers through an R-deep ring of 16-byte buffer loads with no barrier in
// the loop.  Per 32-channel step each wave runs v_mfma_f32_16x16x32_bf16 for
//     S += X Q^T      (the relevance contraction),
//     G += X X^T      (diagonal: |x|^2),
//     P += X I        (identity columns: channel sums of its tokens),
// and one wave per step adds the query's Gram matrix (diagonal: |q_j|^2), so
// norms and pooling cost no vector-ALU work.  The waves' channel sums meet in
// LDS and are added in wave order.  With one slice the workgroup also finishes
// its tokens' a_{t,n}; with several it writes the partial x . q_j and |x|^2.
//
// Vector-ALU path (fp32 inputs, Q < 16 or tiny frames): tiles of up to 32
// tokens over all channels, one wave per token, wave-reduced dot products.
#include <type_traits>

#include "wz_device.h"

namespace wz {
namespace {

constexpr int kKStep = 32;    // channels per MFMA K step (16x16x32)
constexpr int kQMax = 1024;   // validated bound on query tokens

// Per-unit outputs of the streaming pass (layouts in the workspace carve-up).
struct StreamArgs {
  float* s_part;
  float* g_part;
  float* qg_part;
  float* sig_part;
  float* pool_part;
  float* tok_score;  // written here when there is one slice
  int T, N, C, Q, QP, tiles, slices;
};

// ---------------------------------------------------------------------------
// MFMA path
// ---------------------------------------------------------------------------
// NTG: 16-column query tiles per pass over the slice (queries of more tokens
// take several passes); R: depth of the X prefetch ring in 32-channel steps.
template <int NTG, int R>
__global__ __launch_bounds__(kMaxWaves / kTilesPerWave * 64) void k_relevance_mfma(const uint16_t* __restrict__ X,
                                                                                   const uint16_t* __restrict__ query,
                                                                                   int tile_tokens, int kc,
                                                                                   StreamArgs f) {
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
                                                        int tile_tokens, StreamArgs f) {
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
#define WZ_REL_RING 4  // X prefetch depth in 32-channel steps
#endif

template <int NTG>
void launch_mfma(const RelPlan& pl, const void* X, const void* query, const StreamArgs& fa, hipStream_t s) {
  hipLaunchKernelGGL((k_relevance_mfma<NTG, WZ_REL_RING>), dim3(pl.grid), dim3(pl.threads), 0, s,
                     static_cast<const uint16_t*>(X), static_cast<const uint16_t*>(query), pl.tile_tokens, pl.kc,
                     fa);
}

}  // namespace

bool relevance_uses_mfma(const wz_config& c) {
  // two 16-row MFMA tiles per wave, at least 2 waves: frames of at least 49 tokens
  return c.in_dtype == WZ_BF16 && c.Q >= 16 && c.H * c.W >= 49;
}

hipError_t launch_relevance_stream(const wz_config& c, const void* X, const void* query, float* tok_score,
                                   const Workspace& ws, hipStream_t s) {
  const RelPlan pl = relevance_plan(c);
  const StreamArgs fa{ws.s_part, ws.g_part, ws.qg_part, ws.sig_part, ws.pool_part, tok_score, c.T, c.H * c.W,
                      c.C,       c.Q,       qpad(c.Q),  pl.tiles,    pl.slices};
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
