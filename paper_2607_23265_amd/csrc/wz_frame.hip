// Per-frame kernel, one workgroup per frame.  It finishes stage 1 from the
// streaming pass's per-unit partials and prepares the token selection of
// stage 3:
//
//   a_{t,n} = max_j (sum_s S_s[n][j]) / (|q_j| |x_n|)       (several slices;
//             with one slice the streaming pass wrote a_{t,n} itself)
//   r_t     = max_j sigma_j / (|q_j| |p_t|),  sigma_j = p_t . q_j   (Sec. 3.2.1)
//   delta_t = clamp(1 - p_t . p_{t-1} / (|p_t| |p_{t-1}|), 0, 2), delta_0 = 0
//             (Sec. 3.2.2, Eq. (8); the mean's cosine is the sum's)
// with cos := 0 (a = 0, r = 0, delta = 1) when a vector is zero, and
//   rank[t][n] = number of the frame's tokens with a larger score (ties: the
//                smaller index ranks first), so that a frame's n_t kept tokens
//                are those of rank < n_t whatever n_t turns out to be;
//   sal[t][n]  = M_t = min-max of the frame's scores (Eq. (7); 0 when all
//                scores are equal).
// Every partial is added in a fixed order (tile, then slice), so results do
// not depend on timing.  All loads of the partials are issued before the
// first one is used.
//
// Without partials (scores given by the caller) only the preparation runs.
#include "wz_device.h"

namespace wz {
namespace {

constexpr int kQMax = 1024;
constexpr int kThreads = 512;

struct FrameArgs {
  const float* s_part;     // [T][S][N][QP]   (several slices)
  const float* g_part;     // [T][S][N]       (several slices)
  const float* qg_part;    // [T][S][Q]
  const float* sig_part;   // [T][tiles][S][Q]
  const float* pool_part;  // [T][tiles][C]
  float* tok_score;        // [T][N]  in (one slice, or preparation only) or out
  float* frame_rel;        // [T]
  float* frame_delta;      // [T]
  int32_t* rank;           // [T][N]
  float* sal;              // [T][N]
  int T, N, C, Q, QP, tiles, slices;
  int finish;              // 0: scores given, preparation only
};

__global__ __launch_bounds__(kThreads) void k_frame(const FrameArgs f) {
  constexpr int NW = kThreads / kWave;
  constexpr int AV = kTokMax / kThreads;  // tokens per thread at most
  constexpr int U = 4, SB = 4;            // partial-score batch: units x slices per thread
  constexpr int PF = 2;                   // channel-sum vectors per thread issued up front
  __shared__ float s_rq[kQMax];
  __shared__ float s_xn[kTokMax];
  __shared__ uint32_t s_best[kTokMax];
  __shared__ uint64_t s_key[kTokMax];
  __shared__ double s_red[4][NW];
  __shared__ float s_mm[2][NW];

  const int t = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int N = f.N, C = f.C, Q = f.Q, QP = f.QP, S = f.slices, tiles = f.tiles, K = tiles * S, C4 = C / 4;
  float av[AV];  // scores of tokens tid + i * kThreads
  const __amdgpu_buffer_rsrc_t ares = make_rsrc(f.tok_score + size_t(t) * N, uint32_t(N) * 4);

  if (f.finish) {
    const int G4 = QP / 4, units = N * G4;
    const __amdgpu_buffer_rsrc_t sres =
        make_rsrc(f.s_part + size_t(t) * S * N * QP, S > 1 ? uint32_t(S) * N * QP * 4 : 0u);
    const __amdgpu_buffer_rsrc_t qgres = make_rsrc(f.qg_part + size_t(t) * S * Q, uint32_t(S) * Q * 4);
    const __amdgpu_buffer_rsrc_t sgres = make_rsrc(f.sig_part + size_t(t) * K * Q, uint32_t(K) * Q * 4);
    const __amdgpu_buffer_rsrc_t gres = make_rsrc(f.g_part + size_t(t) * S * N, S > 1 ? uint32_t(S) * N * 4 : 0u);
    const __amdgpu_buffer_rsrc_t pbres = make_rsrc(f.pool_part + size_t(t) * tiles * C, uint32_t(tiles) * C * 4);
    const __amdgpu_buffer_rsrc_t pares =
        make_rsrc(f.pool_part + size_t(t > 0 ? t - 1 : 0) * tiles * C, t > 0 ? uint32_t(tiles) * C * 4 : 0u);

    // ---- every first load in flight before any is used ----
    f32x4 v[U][SB];
    auto load_batch = [&](int u0, int s0) {
#pragma unroll
      for (int k = 0; k < U; ++k)
#pragma unroll
        for (int s = 0; s < SB; ++s) {
          const int u = u0 + tid + k * kThreads;
          const bool ok = u < units && s0 + s < S;
          v[k][s] = buf_load_f32x4(sres, ok ? ((s0 + s) * N * QP + u * 4) * 4 : kOOB);
        }
    };
    if (S > 1) load_batch(0, 0);
    if (S == 1) {
#pragma unroll
      for (int i = 0; i < AV; ++i) {
        const int n = tid + i * kThreads;
        av[i] = buf_load_f32(ares, n < N ? n * 4 : kOOB);
      }
    }
    f32x4 pa[PF], pb[PF];  // tile 0 of p_{t-1} and p_t
#pragma unroll
    for (int i = 0; i < PF; ++i) {
      const int c4 = tid + i * kThreads;
      pa[i] = buf_load_f32x4(pares, c4 < C4 ? c4 * 16 : kOOB);
      pb[i] = buf_load_f32x4(pbres, c4 < C4 ? c4 * 16 : kOOB);
    }

    // 1/|q_j|, sigma_j / |q_j|, |x_n| (several slices)
    double rbest = -INFINITY;
    for (int i = tid; i < max(Q, S > 1 ? N : 0); i += kThreads) {
      float qq = 0.f, sg = 0.f, xx = 0.f;
      for (int k0 = 0; k0 < K; k0 += 4) {
        float a[4], b[4], c[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int k = k0 + e;
          a[e] = buf_load_f32(qgres, (i < Q && k < S) ? (k * Q + i) * 4 : kOOB);
          b[e] = buf_load_f32(sgres, (i < Q && k < K) ? (k * Q + i) * 4 : kOOB);
          c[e] = buf_load_f32(gres, (i < N && k < S) ? (k * N + i) * 4 : kOOB);
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
      if (S > 1 && i < N) {
        s_xn[i] = sqrtf(xx);
        s_best[i] = 0u;
      }
    }

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
    __syncthreads();  // also publishes s_rq, s_xn, s_best
    if (tid == 0) {
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

    if (S > 1) {
      // a_{t,n}: unit u = (token n, columns 4g..4g+3), slices added in order
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
#pragma unroll
      for (int i = 0; i < AV; ++i) {
        const int n = tid + i * kThreads;
        if (n < N) {
          const float xn = s_xn[n];
          av[i] = xn > 0.f ? order_value(s_best[n]) / xn : 0.f;
          f.tok_score[size_t(t) * N + n] = av[i];
        }
      }
    }
  }
  if (!f.finish) {
#pragma unroll
    for (int i = 0; i < AV; ++i) {
      const int n = tid + i * kThreads;
      av[i] = buf_load_f32(ares, n < N ? n * 4 : kOOB);
    }
  }

  // ---- selection keys and the saliency range ----
  float lo = INFINITY, hi = -INFINITY;
#pragma unroll
  for (int i = 0; i < AV; ++i) {
    const int n = tid + i * kThreads;
    if (n < N) {
      s_key[n] = sel_key(av[i], n);
      lo = fminf(lo, av[i]);
      hi = fmaxf(hi, av[i]);
    }
  }
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) {
    lo = fminf(lo, __shfl_xor(lo, m, kWave));
    hi = fmaxf(hi, __shfl_xor(hi, m, kWave));
  }
  if (lane == 0) {
    s_mm[0][wave] = lo;
    s_mm[1][wave] = hi;
  }
  __syncthreads();
  lo = s_mm[0][0];
  hi = s_mm[1][0];
#pragma unroll
  for (int w = 1; w < NW; ++w) {
    lo = fminf(lo, s_mm[0][w]);
    hi = fmaxf(hi, s_mm[1][w]);
  }
  const float range = hi - lo;

  // ---- ranks and M: tpt consecutive lanes share a token, each counting the
  // keys of one part of the frame (read as near-broadcasts, 16 per step) ----
  const int tpt = N <= 64 ? 8 : N <= 128 ? 4 : N <= 256 ? 2 : 1;
  const int part = tid % tpt, per_round = kThreads / tpt;
  const int jlen = (N + tpt - 1) / tpt, jb = min(N, part * jlen), je = min(N, jb + jlen);
  for (int n0 = 0; n0 < N; n0 += per_round) {
    const int n = n0 + tid / tpt;
    int r = 0;
    uint64_t kn = 0;
    if (n < N) {
      kn = s_key[n];
      int j = jb;
      for (; j + 16 <= je; j += 16) {
#pragma unroll
        for (int e = 0; e < 16; ++e) r += s_key[j + e] > kn;
      }
      for (; j < je; ++j) r += s_key[j] > kn;
    }
    for (int m = 1; m < tpt; m <<= 1) r += __shfl_xor(r, m, kWave);
    if (n < N && part == 0) {
      f.rank[size_t(t) * N + n] = r;
      const float a = order_value(uint32_t(kn >> 12));
      f.sal[size_t(t) * N + n] = range > 0.f ? (a - lo) / range : 0.f;
    }
  }
}

}  // namespace

hipError_t launch_frame(const wz_config& c, const Workspace& ws, float* tok_score, float* frame_rel,
                        float* frame_delta, bool finish, hipStream_t s) {
  const RelPlan pl = relevance_plan(c);
  const FrameArgs fa{ws.s_part, ws.g_part, ws.qg_part, ws.sig_part, ws.pool_part, tok_score, frame_rel, frame_delta,
                     ws.rank, ws.sal, c.T, c.H * c.W, c.C, c.Q, qpad(c.Q), pl.tiles, pl.slices, finish ? 1 : 0};
  hipLaunchKernelGGL(k_frame, dim3(c.T), dim3(kThreads), 0, s, fa);
  return hipGetLastError();
}

}  // namespace wz
