// Per-frame finish of stage 1, T x (kChunks + 1) workgroups.  Workgroup
// (t, q < kChunks) adds the channel slices' partial dot products of the q-th
// quarter of frame t's tokens in slice order and forms
//   a_{t,n} = max_j (sum_s S_s[n][j]) / (|q_j| |x_n|)     (several slices;
//             with one slice the streaming pass wrote a_{t,n} itself),
// and workgroup (t, kChunks) forms
//   r_t     = max_j sigma_j / (|q_j| |p_t|),  sigma_j = p_t . q_j   (Sec. 3.2.1)
//   delta_t = clamp(1 - p_t . p_{t-1} / (|p_t| |p_{t-1}|), 0, 2), delta_0 = 0
//             (Sec. 3.2.2, Eq. (8); the mean's cosine is the sum's)
// with cos := 0 (a = 0, r = 0, delta = 1) when a vector is zero.  Spreading a
// frame's partials over several workgroups keeps the read of them (4*S*Q
// bytes per token) from running at one CU's share of the bandwidth.  Every
// partial is added in a fixed order, so results do not depend on timing, and
// all first loads are issued before the first one is used.
#include "wz_device.h"

namespace wz {
namespace {

constexpr int kQMax = 1024;
constexpr int kThreads = 256;
constexpr int kChunks = 4;  // token chunks (workgroups) per frame

struct FrameArgs {
  const float* s_part;     // [T][S][N][QP]   (several slices)
  const float* g_part;     // [T][S][N]       (several slices)
  const float* qg_part;    // [T][S][Q]
  const float* sig_part;   // [T][tiles][S][Q]
  const float* pool_part;  // [T][tiles][C]
  float* tok_score;        // [T][N]  out (several slices)
  float* frame_rel;        // [T]
  float* frame_delta;      // [T]
  int T, N, C, Q, QP, tiles, slices;
};

__global__ __launch_bounds__(kThreads) void k_frame_scores(const FrameArgs f) {
  constexpr int NW = kThreads / kWave;
  constexpr int U = 4, SB = 4;  // partial-score batch: units x slices per thread
  constexpr int PF = 4;         // channel-sum vectors per thread issued up front
  __shared__ float s_rq[kQMax];
  __shared__ float s_xn[kTokMax / kChunks];
  __shared__ uint32_t s_best[kTokMax / kChunks];
  __shared__ double s_red[4][NW];

  const int t = blockIdx.x / (kChunks + 1), q = blockIdx.x % (kChunks + 1);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int N = f.N, C = f.C, Q = f.Q, QP = f.QP, S = f.slices, tiles = f.tiles, K = tiles * S, C4 = C / 4;
  const bool lead = q == kChunks;  // this workgroup forms r_t and delta_t (and no scores)
  const int per = (N + kChunks - 1) / kChunks, n0 = lead ? 0 : min(N, q * per), NQ = lead ? 0 : min(N, n0 + per) - n0;
  const bool scores = S > 1;
  const int G4 = QP / 4, units = NQ * G4;

  const __amdgpu_buffer_rsrc_t sres =
      make_rsrc(f.s_part + size_t(t) * S * N * QP, scores ? uint32_t(S) * N * QP * 4 : 0u);
  const __amdgpu_buffer_rsrc_t qgres = make_rsrc(f.qg_part + size_t(t) * S * Q, uint32_t(S) * Q * 4);
  const __amdgpu_buffer_rsrc_t sgres = make_rsrc(f.sig_part + size_t(t) * K * Q, lead ? uint32_t(K) * Q * 4 : 0u);
  const __amdgpu_buffer_rsrc_t gres = make_rsrc(f.g_part + size_t(t) * S * N, scores ? uint32_t(S) * N * 4 : 0u);
  const __amdgpu_buffer_rsrc_t pbres =
      make_rsrc(f.pool_part + size_t(t) * tiles * C, lead ? uint32_t(tiles) * C * 4 : 0u);
  const __amdgpu_buffer_rsrc_t pares =
      make_rsrc(f.pool_part + size_t(t > 0 ? t - 1 : 0) * tiles * C, lead && t > 0 ? uint32_t(tiles) * C * 4 : 0u);

  // ---- every first load in flight before any is used ----
  f32x4 v[U][SB];
  auto load_batch = [&](int u0, int s0) {
#pragma unroll
    for (int k = 0; k < U; ++k)
#pragma unroll
      for (int s = 0; s < SB; ++s) {
        const int u = u0 + tid + k * kThreads;
        const bool ok = scores && u < units && s0 + s < S;
        v[k][s] = buf_load_f32x4(sres, ok ? ((s0 + s) * N * QP + n0 * QP + u * 4) * 4 : kOOB);
      }
  };
  load_batch(0, 0);
  f32x4 pa[PF], pb[PF];  // tile 0 of p_{t-1} and p_t (lead workgroup; zeros elsewhere)
#pragma unroll
  for (int i = 0; i < PF; ++i) {
    const int c4 = tid + i * kThreads;
    pa[i] = buf_load_f32x4(pares, c4 < C4 ? c4 * 16 : kOOB);
    pb[i] = buf_load_f32x4(pbres, c4 < C4 ? c4 * 16 : kOOB);
  }

  // 1/|q_j| and sigma_j / |q_j| (query index i), |x_n| of the chunk (token index i)
  double rbest = -INFINITY;
  for (int i = tid; i < max(Q, scores ? NQ : 0); i += kThreads) {
    float qq = 0.f, sg = 0.f, xx = 0.f;
    for (int k0 = 0; k0 < K; k0 += 4) {
      float a[4], b[4], c[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int k = k0 + e;
        a[e] = buf_load_f32(qgres, (i < Q && k < S) ? (k * Q + i) * 4 : kOOB);
        b[e] = buf_load_f32(sgres, (i < Q && k < K) ? (k * Q + i) * 4 : kOOB);
        c[e] = buf_load_f32(gres, (i < NQ && k < S) ? (k * N + n0 + i) * 4 : kOOB);
      }
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        qq += a[e];
        sg += b[e];
        xx += c[e];
      }
    }
    if (i < Q) {
      const float rq = qq > 0.f ? 1.0f / sqrtf(qq) : 0.f;
      s_rq[i] = rq;
      rbest = fmax(rbest, double(sg) * rq);
    }
    if (scores && i < NQ) {
      s_xn[i] = sqrtf(xx);
      s_best[i] = 0u;
    }
  }

  if (lead) {
    // channel sums p_{t-1} (a) and p_t (b), tiles added in order
    double ab = 0.0, aa = 0.0, bb = 0.0;
    for (int c0 = 0; c0 < C4; c0 += PF * kThreads) {
#pragma unroll
      for (int i = 0; i < PF; ++i) {
        const int c4 = c0 + tid + i * kThreads;
        f32x4 x = pa[i], y = pb[i];
        if (c0 > 0) {
          x = buf_load_f32x4(pares, c4 < C4 ? c4 * 16 : kOOB);
          y = buf_load_f32x4(pbres, c4 < C4 ? c4 * 16 : kOOB);
        }
        for (int k = 1; k < tiles; ++k) {
          x += buf_load_f32x4(pares, c4 < C4 ? (k * C + c4 * 4) * 4 : kOOB);
          y += buf_load_f32x4(pbres, c4 < C4 ? (k * C + c4 * 4) * 4 : kOOB);
        }
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          ab += double(x[e]) * y[e];
          aa += double(x[e]) * x[e];
          bb += double(y[e]) * y[e];
        }
      }
    }
    ab = wave_sum_f64(ab);
    aa = wave_sum_f64(aa);
    bb = wave_sum_f64(bb);
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) rbest = fmax(rbest, __shfl_xor(rbest, m, kWave));
    if (lane == 0) {
      s_red[0][wave] = ab;
      s_red[1][wave] = aa;
      s_red[2][wave] = bb;
      s_red[3][wave] = rbest;
    }
  }
  __syncthreads();  // publishes s_rq, s_xn, s_best and the lead's sums
  if (lead && tid == 0) {
    double sab = 0.0, saa = 0.0, sbb = 0.0, rb = -INFINITY;
    for (int w = 0; w < NW; ++w) {
      sab += s_red[0][w];
      saa += s_red[1][w];
      sbb += s_red[2][w];
      rb = fmax(rb, s_red[3][w]);
    }
    f.frame_rel[t] = float(sbb > 0.0 ? rb / sqrt(sbb) : 0.0);
    double delta = 0.0;
    if (t > 0) delta = (saa > 0.0 && sbb > 0.0) ? fmin(fmax(1.0 - sab / sqrt(saa * sbb), 0.0), 2.0) : 1.0;
    f.frame_delta[t] = float(delta);
  }

  if (scores) {
    // a_{t,n}: unit u = (token n0 + u / G4, columns 4g..4g+3), slices added in order
    for (int u0 = 0; u0 < units; u0 += U * kThreads) {
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
        const int u = u0 + tid + k * kThreads;
        if (u < units) {
          const int n = u / G4, j0 = (u % G4) * 4;
          float m = -INFINITY;
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (j0 + e < Q) m = fmaxf(m, acc[k][e] * s_rq[j0 + e]);
          if (j0 < Q) atomicMax(&s_best[n], order_key(m));
        }
      }
    }
    __syncthreads();
    for (int i = tid; i < NQ; i += kThreads) {
      const float xn = s_xn[i];
      f.tok_score[size_t(t) * N + n0 + i] = xn > 0.f ? order_value(s_best[i]) / xn : 0.f;
    }
  }
}

}  // namespace

hipError_t launch_frame_scores(const wz_config& c, const Workspace& ws, float* tok_score, float* frame_rel,
                               float* frame_delta, hipStream_t s) {
  const RelPlan pl = relevance_plan(c);
  const FrameArgs fa{ws.s_part, ws.g_part, ws.qg_part, ws.sig_part, ws.pool_part, tok_score, frame_rel, frame_delta,
                     c.T,       c.H * c.W, c.C,        c.Q,         qpad(c.Q),    pl.tiles,  pl.slices};
  hipLaunchKernelGGL(k_frame_scores, dim3(c.T * (kChunks + 1)), dim3(kThreads), 0, s, fa);
  return hipGetLastError();
}

}  // namespace wz
