// Stage 2 on its own: the Wavelet Temporal Allocator (Sec. 3.2.2 gate and
// frame filter, Eq. (9)-(11)) and the integer frame budgets (Eq. (16) under
// Eq. (5)) in ONE workgroup: one wave when T <= 64, 256 threads up to
// T = 256, 1024 beyond.  The arithmetic lives in wz_budget.h, which the fused
// selection and gather kernel runs too.
#include "wz_budget.h"

namespace wz {
namespace {

template <int NT, int TV>
__global__ __launch_bounds__(NT) void k_budget(const float* __restrict__ rel, const float* __restrict__ delta,
                                               int T, int N, long long B, int levels, float tau,
                                               int32_t* __restrict__ budget, int32_t* __restrict__ offset,
                                               float* __restrict__ rel_rect) {
  if constexpr (NT == kWave) budget_wave_body(rel, delta, T, N, B, levels, tau, budget, offset, rel_rect);
  else budget_body<NT, TV>(rel, delta, T, N, B, levels, tau, budget, offset, rel_rect);
}

template <int NT, int TV>
void launch_k(const wz_config& c, const float* rel, const float* delta, int32_t* budget, int32_t* offset,
              float* rel_rect, hipStream_t s) {
  hipLaunchKernelGGL((k_budget<NT, TV>), dim3(1), dim3(NT), 0, s, rel, delta, c.T, c.H * c.W, (long long)c.B,
                     c.levels, c.tau, budget, offset, rel_rect);
}

}  // namespace

hipError_t launch_budget(const wz_config& c, const float* frame_rel, const float* frame_delta, int32_t* budget,
                         int32_t* offset, float* rel_rect, hipStream_t s) {
  if (c.T <= 64) launch_k<kWave, 64>(c, frame_rel, frame_delta, budget, offset, rel_rect, s);
  else if (c.T <= 256) launch_k<256, 256>(c, frame_rel, frame_delta, budget, offset, rel_rect, s);
  else launch_k<1024, kTMax>(c, frame_rel, frame_delta, budget, offset, rel_rect, s);
  return hipGetLastError();
}

}  // namespace wz
