// Stage 2 on its own: the Wavelet Temporal Allocator (gate and frame
// filter of Sec. 3.2.2; Sec. 3.2.3, Eq. (9)-(11)) and the integer frame budgets (Sec. 3.2.4, Eq. (16)
// under Eq. (5)) in ONE workgroup: one wave up to T = 256 (every value in
// registers up to 64 frames, four frames per lane in LDS above), 1024
// threads beyond.  The arithmetic lives in wz_budget.h, which the fused
// selection and gather kernel runs too.  With a db4 or bior4.4 temporal basis
// the LDS version runs at every T, with 256 threads from 65 to 256 frames.
#include "wz_budget.h"

namespace wz {
namespace {

struct BudgetArgs {
  const float* rel;
  const float* delta;
  int32_t* budget;
  int32_t* offset;
  float* rel_rect;
};
static_assert(sizeof(VideoArgs<BudgetArgs>) <= 4096, "per-video arguments exceed the kernel argument limit");

// GENERAL: the filter-bank allocator (bank) instead of the Haar one.
template <int NT, int TV, bool GENERAL>
__global__ __launch_bounds__(NT) void k_budget(const VideoArgs<BudgetArgs> va, int T, int N, long long B, int levels,
                                               float tau, const Bank bank) {
  const BudgetArgs& a = va.v[blockIdx.y];
  if constexpr (GENERAL)
    budget_body<NT, TV>(a.rel, a.delta, T, N, B, levels, tau, a.budget, a.offset, a.rel_rect, &bank);
  else if constexpr (NT == kWave && TV == kWave)
    budget_wave_body(a.rel, a.delta, T, N, B, levels, tau, a.budget, a.offset, a.rel_rect);
  else if constexpr (NT == kWave && TV <= 4 * kWave)
    budget_wave_slots<TV>(a.rel, a.delta, T, N, B, levels, tau, a.budget, a.offset, a.rel_rect);
  else
    budget_body<NT, TV>(a.rel, a.delta, T, N, B, levels, tau, a.budget, a.offset, a.rel_rect);
}

template <int NT, int TV>
void launch_k(const wz_config& c, const VideoArgs<BudgetArgs>& va, int V, hipStream_t s) {
  const Bank bank = c.temporal_basis == WZ_HAAR ? Bank{} : make_bank(c.temporal_basis);
  if (c.temporal_basis == WZ_HAAR)
    hipLaunchKernelGGL((k_budget<NT, TV, false>), dim3(1, V), dim3(NT), 0, s, va, c.T, c.H * c.W, (long long)c.B,
                       c.levels, c.tau, bank);
  else
    hipLaunchKernelGGL((k_budget<NT, TV, true>), dim3(1, V), dim3(NT), 0, s, va, c.T, c.H * c.W, (long long)c.B,
                       c.levels, c.tau, bank);
}

}  // namespace

hipError_t launch_budget(const wz_config& c, const float* frame_rel, const float* frame_delta, int32_t* budget,
                         int32_t* offset, float* rel_rect, hipStream_t s, const Videos& vs) {
  VideoArgs<BudgetArgs> va{};
  for (int v = 0; v < vs.V; ++v)
    va.v[v] = BudgetArgs{advance(frame_rel, v * vs.ws), advance(frame_delta, v * vs.ws), advance(budget, v * vs.bud),
                         advance(offset, v * vs.off), advance(rel_rect, v * vs.ws)};
  // (a filter bank's convolutions spread better over four waves)
  if (c.T <= 64) launch_k<kWave, 64>(c, va, vs.V, s);
  else if (c.T <= 128 && c.temporal_basis == WZ_HAAR) launch_k<kWave, 128>(c, va, vs.V, s);
  else if (c.T <= 256 && c.temporal_basis == WZ_HAAR) launch_k<kWave, 256>(c, va, vs.V, s);
  else if (c.T <= 256) launch_k<256, 256>(c, va, vs.V, s);
  else launch_k<1024, kTMax>(c, va, vs.V, s);
  return hipGetLastError();
}

}  // namespace wz
