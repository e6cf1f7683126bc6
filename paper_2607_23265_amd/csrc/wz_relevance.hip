// Stage 1: similarity-branch Cross-Modal Scorer (Sec. 3.2.1) and Visual Change
// Estimator (Sec. 3.2.2, Eq. (8)) in one streaming pass over the frames.
//
// Pass A (k_relevance_mfma / k_relevance_valu) -- one workgroup per tile of up
// to 32 consecutive tokens of one frame, reading every channel of its tokens
// exactly once from HBM.  Per token it produces the saliency
//     a_{t,n} = max_j (x . q_j) / (|x| |q_j|)
// and per tile the channel sums (for the frame's pooled feature) and the
// column sums sum_n x_n . q_j (for the frame relevance).
//
// Pass B (k_frame_reduce) -- one workgroup per frame combines the tile sums
// in a fixed order into the pooled feature p_t = sum_n x_{t,n}, and computes
//     r_t     = max_j (p_t . q_j) / (|p_t| |q_j|)       (mean or sum: same cosine)
//     delta_t = clamp(1 - p_t . p_{t-1} / (|p_t| |p_{t-1}|), 0, 2),  delta_0 = 0
// (cos := 0, so delta = 1, when a pooled feature is zero).
//
// MFMA path (bf16, Q >= 16): the relevance contraction S = X Q^T runs on
// v_mfma_f32_16x16x32_bf16.  Each lane's 16-byte load of 8 consecutive
// channels of one token is the A operand as loaded; the same registers also
// feed a Gram tile X X^T (its diagonal is |x|^2) and an identity tile X I
// (it adds the tile's tokens channel by channel, i.e. the pooled sum), so
// norms and pooling cost no vector-ALU work.  Partial results of the
// workgroup's waves (each wave owns every NW-th block of 32 channels) are
// combined through LDS in a fixed order.
#include "wz_internal.h"

namespace wz {
namespace {

constexpr int kKStep = 32;  // channels per MFMA K step (16x16x32)

__device__ __forceinline__ bf16x8 load_bf16x8(const uint16_t* p) {
  return *reinterpret_cast<const bf16x8*>(p);
}

// Index math of one 16x16 MFMA accumulator (f32x4 per lane): element e of lane
// l is row 4*(l>>4) + e, column l & 15.
template <int MT, int NTG, int NW, int U>
__global__ __launch_bounds__(NW * kWave) void k_relevance_mfma(
    const uint16_t* __restrict__ X, const uint16_t* __restrict__ query, int N, int C, int Q,
    int tiles, int tile_tokens, float* __restrict__ tok_score, float* __restrict__ pool_part,
    float* __restrict__ sig_part, float* __restrict__ rq_out) {
  constexpr int ROWS = MT * 16;
  constexpr int COLS = NTG * 16;
  __shared__ float s_red[NW][ROWS][17];
  __shared__ float s_gpart[NW][ROWS];
  __shared__ float s_qpart[NW][COLS];
  __shared__ float s_rq[COLS];
  __shared__ float s_xn[ROWS];

  const int tile = blockIdx.x % tiles;
  const int t = blockIdx.x / tiles;
  const int tok0 = tile * tile_tokens;
  const int TM = min(tile_tokens, N - tok0);
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int row = lane & 15;
  const int grp = lane >> 4;
  const int ksteps = (C + kKStep - 1) / kKStep;
  const size_t part = size_t(t) * tiles + tile;

  // Identity operands: slot i of the lane with column `row`, K group `grp`
  // holds channel 8*grp + i of the step; I_s selects channel 16*s + column.
  bf16x8 I0, I1;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    I0[i] = (__bf16)((8 * grp + i == row) ? 1.0f : 0.0f);
    I1[i] = (__bf16)((8 * grp + i == 16 + row) ? 1.0f : 0.0f);
  }

  const uint16_t* xrow[MT];
  bool xok[MT];
#pragma unroll
  for (int m = 0; m < MT; ++m) {
    const int r = m * 16 + row;
    xok[m] = r < TM;
    xrow[m] = X + (size_t(t) * N + tok0 + (xok[m] ? r : 0)) * C;
  }

  f32x4 G[MT];
#pragma unroll
  for (int m = 0; m < MT; ++m) G[m] = f32x4{0.f, 0.f, 0.f, 0.f};

  float best = -INFINITY;  // epilogue: running max over j of S * rq for row tid>>2
  const int er = tid >> 2;           // epilogue row
  const int eq = (tid & 3) * 4;      // epilogue first column of the quad
  const bool erow = tid < ROWS * 4;  // thread takes part in the epilogue

  const int groups = (Q + COLS - 1) / COLS;
  for (int g = 0; g < groups; ++g) {
    const int qg0 = g * COLS;
    const uint16_t* qrow[NTG];
    bool qok[NTG];
#pragma unroll
    for (int n = 0; n < NTG; ++n) {
      const int j = qg0 + n * 16 + row;
      qok[n] = j < Q;
      qrow[n] = query + size_t(qok[n] ? j : 0) * C;
    }
    f32x4 S[MT][NTG];
    f32x4 QG[NTG];
#pragma unroll
    for (int n = 0; n < NTG; ++n) {
      QG[n] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int m = 0; m < MT; ++m) S[m][n] = f32x4{0.f, 0.f, 0.f, 0.f};
    }

    for (int ks0 = wave; ks0 < ksteps; ks0 += NW * U) {
      bf16x8 a[U][MT], b[U][NTG];
      const bf16x8 zero = {};
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int ks = ks0 + u * NW;
        const int c = ks * kKStep + grp * 8;
        const bool cok = ks < ksteps && c < C;
#pragma unroll
        for (int m = 0; m < MT; ++m) a[u][m] = (cok && xok[m]) ? load_bf16x8(xrow[m] + c) : zero;
#pragma unroll
        for (int n = 0; n < NTG; ++n) b[u][n] = (cok && qok[n]) ? load_bf16x8(qrow[n] + c) : zero;
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int ks = ks0 + u * NW;
        if (ks >= ksteps) break;
#pragma unroll
        for (int n = 0; n < NTG; ++n) {
#pragma unroll
          for (int m = 0; m < MT; ++m)
            S[m][n] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[u][m], b[u][n], S[m][n], 0, 0, 0);
          QG[n] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(b[u][n], b[u][n], QG[n], 0, 0, 0);
        }
        if (g == 0) {
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
          const int ch = ks * kKStep + lane;
          if (lane < 32 && ch < C) pool_part[part * C + ch] = lane < 16 ? v0 : v1;
        }
      }
    }

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
    if (tid < COLS) {
      float s = 0.f;
#pragma unroll
      for (int w = 0; w < NW; ++w) s += s_qpart[w][tid];
      const float rq = s > 0.f ? 1.0f / sqrtf(s) : 0.f;
      s_rq[tid] = rq;
      if (blockIdx.x == 0 && qg0 + tid < Q) rq_out[qg0 + tid] = rq;
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
          if (j < Q && er < TM) best = fmaxf(best, v * s_rq[n * 16 + eq + k]);
          s_red[0][er][eq + k] = v;
        }
      }
      __syncthreads();
      if (tid < 16) {
        const int j = qg0 + n * 16 + tid;
        if (j < Q) {
          float s = 0.f;
          for (int r = 0; r < TM; ++r) s += s_red[0][r][tid];
          sig_part[part * Q + j] = s;
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
}

// Vector-ALU path (fp32 inputs, or bf16 with fewer than 16 query tokens).
// One wave per token at a time: lanes stride over 16-byte channel vectors,
// the dot products with up to 16 query tokens per pass are wave-reduced.
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

template <typename In, int NW>
__global__ __launch_bounds__(NW * kWave) void k_relevance_valu(
    const In* __restrict__ X, const In* __restrict__ query, int N, int C, int Q, int tiles,
    int tile_tokens, float* __restrict__ tok_score, float* __restrict__ pool_part,
    float* __restrict__ sig_part, float* __restrict__ rq_out) {
  constexpr int V = Vec<In>::kN;
  constexpr int QB = 16;
  __shared__ float s_rq[1024];
  __shared__ float s_sig[NW][1024];

  const int tile = blockIdx.x % tiles;
  const int t = blockIdx.x / tiles;
  const int tok0 = tile * tile_tokens;
  const int TM = min(tile_tokens, N - tok0);
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int nvec = C / V;
  const size_t part = size_t(t) * tiles + tile;

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
  for (int j = tid; j < NW * 1024; j += NW * kWave) (&s_sig[0][0])[j] = 0.f;
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
  for (int v = tid; v < nvec; v += NW * kWave) {
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
    for (int i = 0; i < V; ++i) pool_part[part * C + v * V + i] = acc[i];
  }
  __syncthreads();
  for (int j = tid; j < Q; j += NW * kWave) {
    float s = 0.f;
    for (int w = 0; w < NW; ++w) s += s_sig[w][j];
    sig_part[part * Q + j] = s;
  }
}

// Pass B: per frame, combine the tile sums and derive r_t and delta_t.
// delta = 1 - cos(a, b) is evaluated as |a/|a| - b/|b||^2 / 2, which equals it
// exactly in real arithmetic and avoids the cancellation of 1 - cos when
// adjacent frames are nearly identical.
__global__ __launch_bounds__(256) void k_frame_reduce(const float* __restrict__ pool_part,
                                                      const float* __restrict__ sig_part,
                                                      const float* __restrict__ rq, int C, int Q,
                                                      int tiles, float* __restrict__ frame_rel,
                                                      float* __restrict__ frame_delta) {
  constexpr int kW = 4;
  __shared__ double s_acc[2][kW];
  __shared__ double s_norm[2];
  const int t = blockIdx.x;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const float* cur = pool_part + size_t(t) * tiles * C;
  const float* prv = t > 0 ? pool_part + size_t(t - 1) * tiles * C : nullptr;
  // pass 1: |p_t|^2 and |p_{t-1}|^2 (tile sums added in tile order)
  double pp = 0.0, qq = 0.0;
  for (int c = tid; c < C; c += 256) {
    float p = 0.f;
    for (int k = 0; k < tiles; ++k) p += cur[size_t(k) * C + c];
    pp += double(p) * p;
    if (prv) {
      float p1 = 0.f;
      for (int k = 0; k < tiles; ++k) p1 += prv[size_t(k) * C + c];
      qq += double(p1) * p1;
    }
  }
  pp = wave_sum_f64(pp);
  qq = wave_sum_f64(qq);
  if (lane == 0) { s_acc[0][wave] = pp; s_acc[1][wave] = qq; }
  __syncthreads();
  if (tid == 0) {
    s_norm[0] = sqrt((s_acc[0][0] + s_acc[0][1]) + (s_acc[0][2] + s_acc[0][3]));
    s_norm[1] = sqrt((s_acc[1][0] + s_acc[1][1]) + (s_acc[1][2] + s_acc[1][3]));
  }
  __syncthreads();
  const double na = s_norm[0], nb = s_norm[1];
  // pass 2: |a/|a| - b/|b||^2
  if (prv && na > 0.0 && nb > 0.0) {
    double dd = 0.0;
    for (int c = tid; c < C; c += 256) {
      float p = 0.f, p1 = 0.f;
      for (int k = 0; k < tiles; ++k) p += cur[size_t(k) * C + c];
      for (int k = 0; k < tiles; ++k) p1 += prv[size_t(k) * C + c];
      const double d = double(p) / na - double(p1) / nb;
      dd += d * d;
    }
    dd = wave_sum_f64(dd);
    __syncthreads();
    if (lane == 0) s_acc[0][wave] = dd;
    __syncthreads();
    if (tid == 0) {
      const double delta = 0.5 * ((s_acc[0][0] + s_acc[0][1]) + (s_acc[0][2] + s_acc[0][3]));
      frame_delta[t] = float(fmin(fmax(delta, 0.0), 2.0));
    }
  } else if (tid == 0) {
    frame_delta[t] = t > 0 ? 1.0f : 0.0f;  // a zero pooled feature: cos := 0
  }
  // r_t = max_j sigma_{t,j} / (|p_t| |q_j|)
  double best = -INFINITY;
  for (int j = tid; j < Q; j += 256) {
    float s = 0.f;
    for (int k = 0; k < tiles; ++k) s += sig_part[(size_t(t) * tiles + k) * Q + j];
    const double c = na > 0.0 ? double(s) * rq[j] / na : 0.0;
    best = fmax(best, c);
  }
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) best = fmax(best, __shfl_xor(best, m, kWave));
  __syncthreads();
  if (lane == 0) s_acc[1][wave] = best;
  __syncthreads();
  if (tid == 0)
    frame_rel[t] = float(fmax(fmax(s_acc[1][0], s_acc[1][1]), fmax(s_acc[1][2], s_acc[1][3])));
}

template <int MT, int NTG>
void launch_mfma_variant(const wz_config& c, const Tiling& tl, const void* X, const void* query,
                         float* tok_score, const Workspace& ws, hipStream_t s) {
  constexpr int NW = 4;
  constexpr int U = NTG <= 2 ? 4 : 2;
  const int grid = c.T * tl.tiles_per_frame;
  hipLaunchKernelGGL((k_relevance_mfma<MT, NTG, NW, U>), dim3(grid), dim3(NW * kWave), 0, s,
                     static_cast<const uint16_t*>(X), static_cast<const uint16_t*>(query), c.H * c.W, c.C,
                     c.Q, tl.tiles_per_frame, tl.tile_tokens, tok_score, ws.pool_part, ws.sig_part, ws.rq);
}

template <int MT>
void launch_mfma_mt(const wz_config& c, const Tiling& tl, const void* X, const void* query,
                    float* tok_score, const Workspace& ws, hipStream_t s) {
  const int nt = (c.Q + 15) / 16;
  if (nt <= 1) launch_mfma_variant<MT, 1>(c, tl, X, query, tok_score, ws, s);
  else if (nt <= 2) launch_mfma_variant<MT, 2>(c, tl, X, query, tok_score, ws, s);
  else launch_mfma_variant<MT, 4>(c, tl, X, query, tok_score, ws, s);
}

}  // namespace

bool relevance_uses_mfma(const wz_config& c) { return c.in_dtype == WZ_BF16 && c.Q >= 16; }

hipError_t launch_relevance(const wz_config& c, const void* X, const void* query, float* tok_score,
                            float* frame_rel, float* frame_delta, const Workspace& ws, hipStream_t s) {
  const Tiling tl = relevance_tiling(c);
  const int grid = c.T * tl.tiles_per_frame;
  if (relevance_uses_mfma(c)) {
    if (tl.mtiles == 1) launch_mfma_mt<1>(c, tl, X, query, tok_score, ws, s);
    else launch_mfma_mt<2>(c, tl, X, query, tok_score, ws, s);
  } else if (c.in_dtype == WZ_BF16) {
    hipLaunchKernelGGL((k_relevance_valu<uint16_t, 4>), dim3(grid), dim3(256), 0, s,
                       static_cast<const uint16_t*>(X), static_cast<const uint16_t*>(query), c.H * c.W,
                       c.C, c.Q, tl.tiles_per_frame, tl.tile_tokens, tok_score, ws.pool_part, ws.sig_part,
                       ws.rq);
  } else {
    hipLaunchKernelGGL((k_relevance_valu<float, 4>), dim3(grid), dim3(256), 0, s,
                       static_cast<const float*>(X), static_cast<const float*>(query), c.H * c.W, c.C,
                       c.Q, tl.tiles_per_frame, tl.tile_tokens, tok_score, ws.pool_part, ws.sig_part,
                       ws.rq);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_frame_reduce, dim3(c.T), dim3(256), 0, s, ws.pool_part, ws.sig_part, ws.rq, c.C,
                     c.Q, tl.tiles_per_frame, frame_rel, frame_delta);
  return hipGetLastError();
}

}  // namespace wz
