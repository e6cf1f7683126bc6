// C ABI of the condensation pass: argument validation, workspace carve-up and
// the launch sequence.  Declarations and contracts are in include/wavezip.h.
#include <cmath>
#include <cstdint>
#include <mutex>

#include "wz_internal.h"

using namespace wz;

namespace {

// Scratch for wz_condense_noalloc: a file-scope device array in place of a
// caller's workspace.  Every GPU the library runs on holds its own copy for
// the life of the process.  Host code never uses the array's name as an
// address (on the host it is only a stand-in for the symbol): the device
// address comes from hipGetSymbolAddress, once per device, with that device
// current.
constexpr size_t kScratchBytes = size_t(32) << 20;
__device__ __align__(256) char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch[kMaxDevices] = {};

// Device address of the current device's scratch array (looked up on the
// first call on that device).
wz_status scratch_of_current_device(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return WZ_ERR_DEVICE;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return WZ_ERR_DEVICE;
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  return WZ_OK;
}

}  // namespace

namespace {

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

wz_status check_config(const wz_config* c) {
  if (!c) return WZ_ERR_NULL;
  if ((c->in_dtype != WZ_F32 && c->in_dtype != WZ_BF16) || (c->out_dtype != WZ_F32 && c->out_dtype != WZ_BF16))
    return WZ_ERR_DTYPE;
  if (c->T < 1 || c->T > 2048 || c->H < 1 || c->W < 1 || int64_t(c->H) * c->W > 4096 || c->Q < 1 ||
      c->Q > 1024 || c->C < 8 || c->C > 65536 || c->C % 8 != 0)
    return WZ_ERR_SHAPE;
  if (c->levels < 1 || c->levels > 16 || !std::isfinite(c->lambda_) || c->lambda_ < 0.f ||
      !std::isfinite(c->tau) || c->tau < 0.f || c->tau > 2.f || (c->assign != WZ_SELECT && c->assign != WZ_INTERP) ||
      c->spatial_levels < 0 || c->spatial_levels > 2 || (c->spatial_levels == 2 && c->assign != WZ_SELECT) ||
      c->temporal_basis < WZ_HAAR || c->temporal_basis > WZ_BIOR44 || c->spatial_basis < WZ_HAAR ||
      c->spatial_basis > WZ_BIOR44 || (c->spatial_basis != WZ_HAAR && (c->assign != WZ_SELECT || c->spatial_levels > 1)))
    return WZ_ERR_PARAM;
  if (c->spatial_basis != WZ_HAAR && !filter_assign_supported(*c)) return WZ_ERR_SHAPE;
  if (c->B < 0 || c->B > int64_t(c->T) * c->H * c->W) return WZ_ERR_BUDGET;
  return WZ_OK;
}

wz_status check_ptr(const void* p, uintptr_t align) {
  if (!p) return WZ_ERR_NULL;
  if (!aligned(p, align)) return WZ_ERR_ALIGN;
  return WZ_OK;
}

#define WZ_TRY(expr)                 \
  do {                               \
    const wz_status st_ = (expr);    \
    if (st_ != WZ_OK) return st_;    \
  } while (0)

wz_status from_hip(hipError_t e) { return e == hipSuccess ? WZ_OK : WZ_ERR_DEVICE; }

}  // namespace

namespace {

// The whole pass for V videos of one shape (wz_condense, wz_condense_batch).
// V videos (shared_x false) or V queries over one video (shared_x true);
// split: the workspace layout with the filter-bank operator rows (see
// workspace_layout)
wz_status condense_videos(const wz_config* cfg, int V, bool shared_x, const void* X, const void* query,
                          void* out_tokens, int32_t* out_index, int32_t* budget, int32_t* offset, void* ws,
                          size_t ws_bytes, void* stream, bool split = true) {
  WZ_TRY(check_config(cfg));
  WZ_TRY(check_ptr(X, 16));
  WZ_TRY(check_ptr(query, 16));
  if (cfg->B > 0) {
    WZ_TRY(check_ptr(out_tokens, 16));
    WZ_TRY(check_ptr(out_index, 4));
  }
  if (budget && !aligned(budget, 4)) return WZ_ERR_ALIGN;
  if (offset && !aligned(offset, 4)) return WZ_ERR_ALIGN;
  if (!ws) return WZ_ERR_NULL;
  const Workspace w = workspace_layout(*cfg, static_cast<char*>(ws), split);
  if (!aligned(ws, 256) || ws_bytes / size_t(V) < w.bytes) return WZ_ERR_WORKSPACE;
  const int s_in = cfg->in_dtype == WZ_BF16 ? 2 : 4, s_out = cfg->out_dtype == WZ_BF16 ? 2 : 4;
  const long long TN = (long long)cfg->T * cfg->H * cfg->W;
  Videos vs;
  vs.V = V;
  vs.shared_x = shared_x;
  vs.x = shared_x ? 0 : TN * cfg->C * s_in;
  vs.q = (long long)cfg->Q * cfg->C * s_in;
  vs.ws = (long long)w.bytes;
  vs.out = cfg->B * cfg->C * s_out;
  vs.idx = cfg->B * 4;
  hipStream_t s = static_cast<hipStream_t>(stream);
  // the per-frame kernel also ranks every frame's tokens (for a filter-bank
  // spatial basis its block gates go unused)
  const bool filt = cfg->spatial_basis != WZ_HAAR;
  WZ_TRY(from_hip(launch_relevance_stream(*cfg, X, query, w.tok_score, w, s, vs)));
  WZ_TRY(from_hip(launch_frame(*cfg, w, w.tok_score, w.frame_rel, w.frame_delta, true, s, vs)));
  vs.bud = budget ? (long long)cfg->T * 4 : vs.ws;
  vs.off = offset ? ((long long)cfg->T + 1) * 4 : vs.ws;
  if (cfg->T <= kFusedTMax && cfg->temporal_basis == WZ_HAAR && !filt) {  // budgets inside the selection kernel
    vs.bud = (long long)cfg->T * 4;
    vs.off = ((long long)cfg->T + 1) * 4;
    return from_hip(launch_assign_gather(*cfg, X, w.tok_score, w.frame_rel, w.frame_delta, nullptr, &w, budget,
                                         offset, out_tokens, out_index, s, vs));
  }
  int32_t* bud = budget ? budget : w.budget;
  int32_t* off = offset ? offset : w.offset;
  if (filt && filter_budget_folds(*cfg))  // budgets inside the modulator's first kernel
    return from_hip(launch_filter_assign(*cfg, X, w.tok_score, nullptr, w.rank, w.frows, out_tokens, out_index, s, vs,
                                         FoldedBudget{w.frame_rel, w.frame_delta, bud, off}));
  WZ_TRY(from_hip(launch_budget(*cfg, w.frame_rel, w.frame_delta, bud, off, nullptr, s, vs)));
  if (filt)
    return from_hip(launch_filter_assign(*cfg, X, w.tok_score, off, w.rank, w.frows, out_tokens, out_index, s, vs));
  return from_hip(launch_assign_gather(*cfg, X, w.tok_score, nullptr, nullptr, off, &w, nullptr, nullptr, out_tokens,
                                       out_index, s, vs));
}

}  // namespace

extern "C" {

size_t wz_workspace_bytes(const wz_config* cfg) {
  if (check_config(cfg) != WZ_OK) return 0;
  return workspace_layout(*cfg, nullptr).bytes;
}

const char* wz_status_str(wz_status s) {
  switch (s) {
    case WZ_OK: return "WZ_OK";
    case WZ_ERR_NULL: return "WZ_ERR_NULL: a required pointer is NULL";
    case WZ_ERR_ALIGN: return "WZ_ERR_ALIGN: a pointer is not suitably aligned";
    case WZ_ERR_SHAPE: return "WZ_ERR_SHAPE: a dimension is out of the supported range";
    case WZ_ERR_DTYPE: return "WZ_ERR_DTYPE: unknown data type";
    case WZ_ERR_PARAM: return "WZ_ERR_PARAM: levels, lambda or tau out of range";
    case WZ_ERR_BUDGET: return "WZ_ERR_BUDGET: B must satisfy 0 <= B <= T*H*W";
    case WZ_ERR_WORKSPACE: return "WZ_ERR_WORKSPACE: workspace too small or misaligned";
    case WZ_ERR_DEVICE: return "WZ_ERR_DEVICE: a HIP call or kernel launch failed";
    case WZ_ERR_SCRATCH:
      return "WZ_ERR_SCRATCH: the problem needs more scratch than wz_condense_noalloc's 32 MiB (use wz_condense)";
  }
  return "unknown wz_status";
}

wz_status wz_relevance(const wz_config* cfg, const void* X, const void* query, float* tok_score,
                       float* frame_rel, float* frame_delta, void* ws, size_t ws_bytes, void* stream) {
  WZ_TRY(check_config(cfg));
  WZ_TRY(check_ptr(X, 16));
  WZ_TRY(check_ptr(query, 16));
  WZ_TRY(check_ptr(tok_score, 4));
  WZ_TRY(check_ptr(frame_rel, 4));
  WZ_TRY(check_ptr(frame_delta, 4));
  if (!ws) return WZ_ERR_NULL;
  const Workspace w = workspace_layout(*cfg, static_cast<char*>(ws));
  if (!aligned(ws, 256) || ws_bytes < w.bytes) return WZ_ERR_WORKSPACE;
  hipStream_t s = static_cast<hipStream_t>(stream);
  WZ_TRY(from_hip(launch_relevance_stream(*cfg, X, query, tok_score, w, s)));
  return from_hip(launch_frame(*cfg, w, tok_score, frame_rel, frame_delta, false, s));
}

wz_status wz_relevance_pass(const wz_config* cfg, const void* X, const void* query, float* tok_score, void* ws,
                            size_t ws_bytes, void* stream) {
  WZ_TRY(check_config(cfg));
  WZ_TRY(check_ptr(X, 16));
  WZ_TRY(check_ptr(query, 16));
  WZ_TRY(check_ptr(tok_score, 4));
  if (!ws) return WZ_ERR_NULL;
  const Workspace w = workspace_layout(*cfg, static_cast<char*>(ws));
  if (!aligned(ws, 256) || ws_bytes < w.bytes) return WZ_ERR_WORKSPACE;
  return from_hip(launch_relevance_stream(*cfg, X, query, tok_score, w, static_cast<hipStream_t>(stream)));
}

wz_status wz_temporal_budget(const wz_config* cfg, const float* frame_rel, const float* frame_delta,
                             int32_t* budget, int32_t* offset, float* rel_rect, void* stream) {
  WZ_TRY(check_config(cfg));
  WZ_TRY(check_ptr(frame_rel, 4));
  WZ_TRY(check_ptr(frame_delta, 4));
  WZ_TRY(check_ptr(budget, 4));
  WZ_TRY(check_ptr(offset, 4));
  if (rel_rect && !aligned(rel_rect, 4)) return WZ_ERR_ALIGN;
  return from_hip(launch_budget(*cfg, frame_rel, frame_delta, budget, offset, rel_rect,
                                static_cast<hipStream_t>(stream)));
}

wz_status wz_spatial_dwt_condense(const wz_config* cfg, const void* X, const float* tok_score,
                                  const int32_t* offset, void* out_tokens, int32_t* out_index, void* stream) {
  WZ_TRY(check_config(cfg));
  WZ_TRY(check_ptr(X, 16));
  WZ_TRY(check_ptr(tok_score, 4));
  WZ_TRY(check_ptr(offset, 4));
  if (cfg->B > 0) {
    WZ_TRY(check_ptr(out_tokens, 16));
    WZ_TRY(check_ptr(out_index, 4));
  }
  if (cfg->spatial_basis != WZ_HAAR)
    return from_hip(
        launch_filter_assign(*cfg, X, tok_score, offset, nullptr, nullptr, out_tokens, out_index,
                             static_cast<hipStream_t>(stream)));
  return from_hip(launch_assign_gather(*cfg, X, tok_score, nullptr, nullptr, offset, nullptr, nullptr, nullptr,
                                       out_tokens, out_index, static_cast<hipStream_t>(stream)));
}

wz_status wz_condense(const wz_config* cfg, const void* X, const void* query, void* out_tokens,
                      int32_t* out_index, int32_t* budget, int32_t* offset, void* ws, size_t ws_bytes,
                      void* stream) {
  return condense_videos(cfg, 1, false, X, query, out_tokens, out_index, budget, offset, ws, ws_bytes, stream);
}

size_t wz_noalloc_scratch_bytes(void) { return kScratchBytes; }

wz_status wz_condense_noalloc(const wz_config* cfg, const void* X, const void* query, void* out_tokens,
                              int32_t* out_index, int32_t* budget, int32_t* offset, void* stream) {
  WZ_TRY(check_config(cfg));
  // the filter-bank operator rows in the scratch if they fit, else the
  // modulator's fused form (the same rows bit for bit, kept in LDS)
  const bool split = workspace_layout(*cfg, nullptr, true).bytes <= kScratchBytes;
  if (!split && workspace_layout(*cfg, nullptr, false).bytes > kScratchBytes) return WZ_ERR_SCRATCH;
  void* ws = nullptr;
  WZ_TRY(scratch_of_current_device(&ws));
  return condense_videos(cfg, 1, false, X, query, out_tokens, out_index, budget, offset, ws, kScratchBytes, stream,
                         split);
}

wz_status wz_condense_batch(const wz_config* cfg, int32_t videos, const void* X, const void* query,
                            void* out_tokens, int32_t* out_index, int32_t* budget, int32_t* offset, void* ws,
                            size_t ws_bytes, void* stream) {
  if (videos < 1 || videos > kMaxVideos) return WZ_ERR_SHAPE;
  return condense_videos(cfg, videos, false, X, query, out_tokens, out_index, budget, offset, ws, ws_bytes,
                         stream);
}

wz_status wz_condense_queries(const wz_config* cfg, int32_t queries, const void* X, const void* query,
                              void* out_tokens, int32_t* out_index, int32_t* budget, int32_t* offset, void* ws,
                              size_t ws_bytes, void* stream) {
  if (queries < 1 || queries > kMaxVideos) return WZ_ERR_SHAPE;
  return condense_videos(cfg, queries, true, X, query, out_tokens, out_index, budget, offset, ws, ws_bytes,
                         stream);
}

}  // extern "C"
