// Plain streaming read of a device buffer (include/wavezip_probe.h): the
// achievable read rate the pass over the frames is measured against.  Grid
// of 4096 workgroups x 256 threads; each thread reads 16-byte vectors with a
// grid stride, eight loads in flight, and folds them into one word that is
// stored only if it equals an unlikely constant (so the loads stay live).
#include "wz_device.h"
#include "wavezip_probe.h"

namespace wz {
namespace {

constexpr int kProbeGrid = 4096;
constexpr int kProbeThreads = 256;
constexpr int kProbeDepth = 8;

__global__ __launch_bounds__(kProbeThreads) void k_stream_read(const u32x4* __restrict__ x, size_t nvec,
                                                               uint32_t* sink) {
  const size_t stride = size_t(gridDim.x) * blockDim.x;
  size_t i = size_t(blockIdx.x) * blockDim.x + threadIdx.x;
  uint32_t acc = 0;
  for (; i + (kProbeDepth - 1) * stride < nvec; i += kProbeDepth * stride) {
    u32x4 v[kProbeDepth];
#pragma unroll
    for (int u = 0; u < kProbeDepth; ++u) v[u] = __builtin_nontemporal_load(&x[i + u * stride]);
#pragma unroll
    for (int u = 0; u < kProbeDepth; ++u) acc ^= v[u][0] ^ v[u][1] ^ v[u][2] ^ v[u][3];
  }
  for (; i < nvec; i += stride) {
    const u32x4 v = x[i];
    acc ^= v[0] ^ v[1] ^ v[2] ^ v[3];
  }
  if (acc == 0x9E3779B9u) sink[blockIdx.x] = acc;
}

}  // namespace
}  // namespace wz

extern "C" wz_status wz_probe_stream_read(const void* data, size_t bytes, uint32_t* sink, void* stream) {
  if (!data || !sink) return WZ_ERR_NULL;
  if ((reinterpret_cast<uintptr_t>(data) & 15) || (reinterpret_cast<uintptr_t>(sink) & 3)) return WZ_ERR_ALIGN;
  if (bytes % 16) return WZ_ERR_SHAPE;
  hipLaunchKernelGGL(wz::k_stream_read, dim3(wz::kProbeGrid), dim3(wz::kProbeThreads), 0,
                     static_cast<hipStream_t>(stream), static_cast<const wz::u32x4*>(data), bytes / 16, sink);
  return hipGetLastError() == hipSuccess ? WZ_OK : WZ_ERR_DEVICE;
}
