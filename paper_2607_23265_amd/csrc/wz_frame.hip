// Per-frame finish of stage 1, and the selection order of stage 3, in one
// launch with up to two workgroups per frame t:
//   scores  a_{t,n} = max_j (sum_s S_s[n][j]) / (|q_j| |x_n|)   (several
//           channel slices; with one slice the streaming pass wrote a_{t,n}
//           itself), the slices' partials added in slice order;
//   order   the frame's selection ranks and block gates (wz_rank.h), from the
//           scores just formed or read back, written for the selection and
//           gather kernel (the whole pass only);
//   lead    r_t     = max_j sigma_j / (|q_j| |p_t|),  sigma_j = p_t . q_j
//           delta_t = clamp(1 - p_t . p_{t-1} / (|p_t| |p_{t-1}|), 0, 2),
//           delta_0 = 0 (Sec. 3.2.1; Sec. 3.2.2, Eq. (8); the mean's cosine
//           is the sum's), cos := 0 (a = 0, r = 0, delta = 1) when a vector
//           is zero.
// The scores and the order share a workgroup (the order needs every score of
// the frame; 1024 threads when the scores come from several slices' partials,
// else 256).  The lead has its own workgroup, placed on the
// XCD whose workgroups wrote the frame's partial channel sums.  Every partial
// is added in a fixed order, so results do not depend on timing, and first
// loads are issued before the first one is used.
#include "wz_rank.h"

namespace wz {
namespace {

constexpr int kQMax = 1024;
constexpr int kPartThreads = 1024;  // workgroup size when scores come from slice partials
constexpr int kThreads = 256;       // otherwise

struct FrameArgs {
  const float* s_part;     // [T][S][N][QP]   (several slices)
  const float* g_part;     // [T][S][N]       (several slices)
  const float* qg_part;    // [T][S][Q]
  const float* sig_part;   // [T][tiles][S][Q]
  const float* pool_part;  // [T][tiles][C]
  float* tok_score;        // [T][N]  out (several slices), in (one slice)
  float* frame_rel;        // [T]
  float* frame_delta;      // [T]
  int32_t* rank;           // [T][N]  out (order role)
  int32_t* byrank;         // [T][N]
  float* gate;             // [T][N]
  float* gate2;            // [T][N] level-2 gates, or null (one spatial level)
  int T, N, H, W, C, Q, QP, tiles, slices;
  int order;               // the order role runs
  int roles;               // workgroups per frame: 1 + (scores or order role)
  float lam;
};
static_assert(sizeof(VideoArgs<FrameArgs>) <= 4096, "per-video arguments exceed the kernel argument limit");

// scores (and order) of frame t
template <int NTH>
__device__ void scores_role(const FrameArgs& f, int t) {
  constexpr int kNW = NTH / kWave;
  constexpr int TPT = 4;   // threads per token
  constexpr int LB = 8;    // partial-score vectors in flight per thread
  __shared__ float s_rq[kQMax];
  __shared__ float s_mm[2 * kNW];
  __shared__ int s_start[kBins], s_fill[kBins];
  extern __shared__ __align__(16) char s_dyn[];
  const int N = f.N, Q = f.Q, QP = f.QP, S = f.slices, G4 = QP / 4;
  const int tid = threadIdx.x;
  RankLds rl;
  rl.key = reinterpret_cast<uint64_t*>(s_dyn);
  rl.rank = reinterpret_cast<int32_t*>(rl.key + N);
  rl.byrank = rl.rank + N;
  rl.gate = reinterpret_cast<float*>(rl.byrank + N);
  rl.order = reinterpret_cast<int32_t*>(rl.gate + N);
  rl.gate2 = f.gate2 ? reinterpret_cast<float*>(rl.order + N) : nullptr;
  rl.start = s_start;
  rl.fill = s_fill;
  rl.mm = s_mm;
  float lo = INFINITY, hi = -INFINITY;

  if (S == 1) {
    if (!f.order) return;
    const __amdgpu_buffer_rsrc_t ares = make_rsrc(f.tok_score + size_t(t) * N, uint32_t(N) * 4);
    for (int n0 = 0; n0 < N; n0 += 4 * NTH) {
      float av[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int n = n0 + u * NTH + tid;
        av[u] = buf_load_f32(ares, n < N ? n * 4 : kOOB);
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int n = n0 + u * NTH + tid;
        if (n < N) {
          rl.key[n] = sel_key(av[u], n);
          lo = fminf(lo, av[u]);
          hi = fmaxf(hi, av[u]);
        }
      }
    }
  } else {
    // token n = n0 + tid / TPT; thread part p takes column groups p, p + TPT, ...
    // in (group, slice) order: item i -> group p + TPT * (i / S), slice i % S
    const __amdgpu_buffer_rsrc_t sres = make_rsrc(f.s_part + size_t(t) * S * N * QP, uint32_t(S) * N * QP * 4);
    const __amdgpu_buffer_rsrc_t gres = make_rsrc(f.g_part + size_t(t) * S * N, uint32_t(S) * N * 4);
    const int part = tid % TPT;
    const int ng = part < G4 ? (G4 - part + TPT - 1) / TPT : 0, items = ng * S;
    auto item_off = [&](int n, int i) {
      const int g = part + TPT * (i / S), s = i % S;
      return (n < N && i < items) ? ((s * N + n) * QP + 4 * g) * 4 : kOOB;
    };
    f32x4 v[LB];
    {
      const int n = tid / TPT;
#pragma unroll
      for (int k = 0; k < LB; ++k) v[k] = buf_load_f32x4(sres, item_off(n, k));
    }
    // |x_n|^2 partials of the first round (thread part 0 of each token) and
    // 1 / |q_j|: slices added in order, every load issued before the sums
    constexpr int SB = 8;  // slices per batch
    const __amdgpu_buffer_rsrc_t qgres = make_rsrc(f.qg_part + size_t(t) * S * Q, uint32_t(S) * Q * 4);
    float gx[SB];
    auto load_g = [&](int n, int s0) {
#pragma unroll
      for (int k = 0; k < SB; ++k)
        gx[k] = buf_load_f32(gres, (part == 0 && n < N && s0 + k < S) ? ((s0 + k) * N + n) * 4 : kOOB);
    };
    load_g(tid / TPT, 0);
    for (int j = tid; j < Q; j += NTH) {
      float qq = 0.f;
      for (int s0 = 0; s0 < S; s0 += SB) {
        float qv[SB];
#pragma unroll
        for (int k = 0; k < SB; ++k) qv[k] = buf_load_f32(qgres, s0 + k < S ? ((s0 + k) * Q + j) * 4 : kOOB);
#pragma unroll
        for (int k = 0; k < SB; ++k)
          if (s0 + k < S) qq += qv[k];
      }
      s_rq[j] = qq > 0.f ? 1.0f / sqrtf(qq) : 0.f;
    }
    lds_barrier();
    for (int n0 = 0; n0 < N; n0 += NTH / TPT) {
      const int n = n0 + tid / TPT;
      if (n0 > 0) {
#pragma unroll
        for (int k = 0; k < LB; ++k) v[k] = buf_load_f32x4(sres, item_off(n, k));
        load_g(n, 0);
      }
      float xx = 0.f;
      for (int s0 = 0; s0 < S; s0 += SB) {
        if (s0 > 0) load_g(n, s0);
#pragma unroll
        for (int k = 0; k < SB; ++k)
          if (s0 + k < S) xx += gx[k];
      }
      float best = -INFINITY;
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
      for (int i0 = 0; i0 < items; i0 += LB) {
        if (i0 > 0) {
#pragma unroll
          for (int k = 0; k < LB; ++k) v[k] = buf_load_f32x4(sres, item_off(n, i0 + k));
        }
#pragma unroll
        for (int k = 0; k < LB; ++k) {
          const int i = i0 + k;
          if (i < items) {
            acc += v[k];
            if (i % S == S - 1) {  // group complete: its columns' scaled scores
              const int j0 = 4 * (part + TPT * (i / S));
#pragma unroll
              for (int e = 0; e < 4; ++e)
                if (j0 + e < Q) best = fmaxf(best, acc[e] * s_rq[j0 + e]);
              acc = f32x4{0.f, 0.f, 0.f, 0.f};
            }
          }
        }
      }
      // the token's four threads are adjacent lanes: max and |x|^2 by DPP
      best = fmaxf(best, __uint_as_float(__builtin_amdgcn_update_dpp(0u, __float_as_uint(best), 0xB1, 0xF, 0xF, false)));
      best = fmaxf(best, __uint_as_float(__builtin_amdgcn_update_dpp(0u, __float_as_uint(best), 0x4E, 0xF, 0xF, false)));
      xx = __uint_as_float(__builtin_amdgcn_update_dpp(0u, __float_as_uint(xx), 0x00, 0xF, 0xF, false));  // lane 0 of the quad
      if (n < N && part == 0) {
        const float xn = sqrtf(xx);
        const float a = xn > 0.f ? best / xn : 0.f;
        f.tok_score[size_t(t) * N + n] = a;
        rl.key[n] = sel_key(a, n);
        lo = fminf(lo, a);
        hi = fmaxf(hi, a);
      }
    }
  }
  if (!f.order) return;
  rank_frame<NTH>(N, f.H, f.W, f.lam, lo, hi, rl);
  lds_barrier();
  for (int n = tid; n < N; n += NTH) {
    f.rank[size_t(t) * N + n] = rl.rank[n];
    f.byrank[size_t(t) * N + n] = rl.byrank[n];
    f.gate[size_t(t) * N + n] = rl.gate[n];
    if (f.gate2) f.gate2[size_t(t) * N + n] = rl.gate2[n];
  }
}

// r_t and delta_t of frame t
template <int NTH>
__device__ void lead_role(const FrameArgs& f, int t) {
  constexpr int kNW = NTH / kWave;
  // tiles of the channel sums loaded at once (1024 threads: every tile of a
  // frame split into up to 8, one vector each, so the reads take one round)
  constexpr int TB = NTH <= 256 ? 4 : 8;
  __shared__ double s_red[4][kNW];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int C = f.C, Q = f.Q, S = f.slices, tiles = f.tiles, K = tiles * S, C4 = C / 4;
  const __amdgpu_buffer_rsrc_t pbres = make_rsrc(f.pool_part + size_t(t) * tiles * C, uint32_t(tiles) * C * 4);
  const __amdgpu_buffer_rsrc_t pares =
      make_rsrc(f.pool_part + size_t(t > 0 ? t - 1 : 0) * tiles * C, t > 0 ? uint32_t(tiles) * C * 4 : 0u);
  const __amdgpu_buffer_rsrc_t qgres = make_rsrc(f.qg_part + size_t(t) * S * Q, uint32_t(S) * Q * 4);
  const __amdgpu_buffer_rsrc_t sgres = make_rsrc(f.sig_part + size_t(t) * K * Q, uint32_t(K) * Q * 4);

  // channel sums p_{t-1} (a) and p_t (b) of channel vectors c4 + NTH * i, i < PF:
  // tiles added in order, the loads of TB tiles of all PF vectors in flight at once
  constexpr int PF = NTH <= 256 ? 4 : 1;
  auto sums = [&](int c4, f32x4 (&x)[PF], f32x4 (&y)[PF]) {
#pragma unroll
    for (int i = 0; i < PF; ++i) x[i] = y[i] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int k0 = 0; k0 < tiles; k0 += TB) {
      f32x4 xa[PF][TB], yb[PF][TB];
#pragma unroll
      for (int i = 0; i < PF; ++i)
#pragma unroll
        for (int k = 0; k < TB; ++k) {
          const int c = c4 + NTH * i;
          const int off = (c < C4 && k0 + k < tiles) ? ((k0 + k) * C + c * 4) * 4 : kOOB;
          xa[i][k] = buf_load_f32x4(pares, off);
          yb[i][k] = buf_load_f32x4(pbres, off);
        }
#pragma unroll
      for (int i = 0; i < PF; ++i)
#pragma unroll
        for (int k = 0; k < TB; ++k) {
          if (k0 + k < tiles) {
            x[i] += xa[i][k];
            y[i] += yb[i][k];
          }
        }
    }
  };
  // sigma_j / |q_j| for query j
  double rbest = -INFINITY;
  for (int j = tid; j < Q; j += NTH) {
    float qq = 0.f, sg = 0.f;
    for (int k0 = 0; k0 < K; k0 += 4) {
      float a[4], b[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int k = k0 + e;
        a[e] = buf_load_f32(qgres, k < S ? (k * Q + j) * 4 : kOOB);
        b[e] = buf_load_f32(sgres, k < K ? (k * Q + j) * 4 : kOOB);
      }
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        qq += a[e];
        sg += b[e];
      }
    }
    const float rq = qq > 0.f ? 1.0f / sqrtf(qq) : 0.f;
    rbest = fmax(rbest, double(sg) * rq);
  }
  double ab = 0.0, aa = 0.0, bb = 0.0;
  for (int c4 = tid; c4 < C4; c4 += PF * NTH) {
    f32x4 x[PF], y[PF];
    sums(c4, x, y);
#pragma unroll
    for (int i = 0; i < PF; ++i)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        ab += double(x[i][e]) * y[i][e];
        aa += double(x[i][e]) * x[i][e];
        bb += double(y[i][e]) * y[i][e];
      }
  }
  auto add = [](double x, double y) { return x + y; };
  ab = wave_reduce_f64(ab, add);
  aa = wave_reduce_f64(aa, add);
  bb = wave_reduce_f64(bb, add);
  rbest = wave_reduce_f64(rbest, [](double x, double y) { return fmax(x, y); });
  if (lane == 0) {
    s_red[0][wave] = ab;
    s_red[1][wave] = aa;
    s_red[2][wave] = bb;
    s_red[3][wave] = rbest;
  }
  lds_barrier();
  if (tid == 0) {
    double sab = 0.0, saa = 0.0, sbb = 0.0, rb = -INFINITY;
    for (int w = 0; w < kNW; ++w) {
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
}

// Workgroup b: frame t = (b / 8 / roles) * 8 + b % 8 (so every workgroup of a
// frame runs on the XCD that streamed it), role (b / 8) % roles; the last role
// is the lead.
template <int NTH>
__global__ __launch_bounds__(NTH) void k_frame(const VideoArgs<FrameArgs> va) {
  const FrameArgs& f = va.v[blockIdx.y];
  const int b = blockIdx.x, xcd = b % kXcds, slot = b / kXcds;
  const int t = (slot / f.roles) * kXcds + xcd, role = slot % f.roles;
  if (t >= f.T) return;
  if (role == f.roles - 1) lead_role<NTH>(f, t);
  else scores_role<NTH>(f, t);
}

}  // namespace

hipError_t launch_frame(const wz_config& c, const Workspace& ws, float* tok_score, float* frame_rel,
                        float* frame_delta, bool order, hipStream_t s, const Videos& vs) {
  const RelPlan pl = relevance_plan(c);
  const int N = c.H * c.W;
  const int roles = (pl.slices > 1 || order) ? 2 : 1;
  // queries sharing one pass over X find the video's channel sums in the first workspace
  const bool shared = vs.shared_x && shared_pass(c, vs.V);
  VideoArgs<FrameArgs> va{};
  for (int v = 0; v < vs.V; ++v) {
    const Workspace w = advance(ws, v * vs.ws);
    va.v[v] = FrameArgs{w.s_part,   w.g_part,  w.qg_part,
                        w.sig_part, shared ? ws.pool_part : w.pool_part, advance(tok_score, v * vs.ws),
                        advance(frame_rel, v * vs.ws), advance(frame_delta, v * vs.ws), w.rank,
                        w.byrank,   w.gate,    c.spatial_levels == 2 && order ? w.gate2 : nullptr, c.T,
                        N,          c.H,       c.W,
                        c.C,        c.Q,       qpad(c.Q),
                        pl.tiles,   pl.slices, order ? 1 : 0,
                        roles,      c.lambda_};
  }
  // key 8 B; rank, byrank, gate, bin order (and level-2 gate) 4 B
  const size_t lds = roles == 2 ? size_t(N) * (c.spatial_levels == 2 ? 28 : 24) : 0;
  const dim3 grid((c.T + kXcds - 1) / kXcds * kXcds * roles, vs.V);
  // 1024 threads when the scores come from slice partials, or when frames
  // are split into many tiles (few frames: the lead's reads spread over more
  // threads and go out in one round)
  if (pl.slices > 1 || pl.tiles >= 8) hipLaunchKernelGGL((k_frame<kPartThreads>), grid, dim3(kPartThreads), lds, s, va);
  else hipLaunchKernelGGL((k_frame<kThreads>), grid, dim3(kThreads), lds, s, va);
  return hipGetLastError();
}

}  // namespace wz
