// Device helpers shared by the gfx950 kernels: raw buffer-resource accesses.
#pragma once

#include <type_traits>

#include "wz_internal.h"

namespace wz {

// Buffer-resource accesses: an offset at or past the resource's size reads
// zeros / drops the write without touching memory, so pad rows and ragged
// edges need no branch (a branch around a load makes the compiler wait for
// every load in flight before the branch joins).
constexpr int kOOB = 0x40000000;       // byte offset beyond any resource here
constexpr int kBufWord3 = 0x00020000;  // gfx9-family raw buffer descriptor word 3

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, int(bytes), kBufWord3);
}
// Same, with base and size passed through readfirstlane: for values the
// compiler cannot prove wave-uniform, a descriptor in VGPRs would turn every
// access into a waterfall loop.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc_uniform(const void* base, uint32_t bytes) {
  const uint64_t a = reinterpret_cast<uint64_t>(base);
  const uint32_t lo = __builtin_amdgcn_readfirstlane(uint32_t(a)), hi = __builtin_amdgcn_readfirstlane(uint32_t(a >> 32));
  const void* p = reinterpret_cast<const void*>((uint64_t(hi) << 32) | lo);
  return make_rsrc(p, __builtin_amdgcn_readfirstlane(bytes));
}
__device__ __forceinline__ bf16x8 buf_load_bf16x8(__amdgpu_buffer_rsrc_t r, int off) {
  return __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
}
__device__ __forceinline__ u32x4 buf_load_u32x4(__amdgpu_buffer_rsrc_t r, int off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
}
__device__ __forceinline__ f32x4 buf_load_f32x4(__amdgpu_buffer_rsrc_t r, int off) {
  return __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
}
__device__ __forceinline__ float buf_load_f32(__amdgpu_buffer_rsrc_t r, int off) {
  return __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0));
}
__device__ __forceinline__ int buf_load_i32(__amdgpu_buffer_rsrc_t r, int off) {
  return int(__builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0));
}
__device__ __forceinline__ void buf_store_f32(float v, __amdgpu_buffer_rsrc_t r, int off) {
  __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v), r, off, 0, 0);
}
// Stores of results that this kernel does not read back, written through the
// L2 to memory (system-coherent, sc1): they do not sit dirty in the L2 until
// the end of the kernel, whose write-back otherwise delays the next kernel by
// about 0.15 us per MB.
constexpr int kWriteThrough = 16;  // buffer-store cache policy: sc1
__device__ __forceinline__ void buf_store_wt_b128(u32x4 v, __amdgpu_buffer_rsrc_t r, int off) {
  __builtin_amdgcn_raw_buffer_store_b128(v, r, off, 0, kWriteThrough);
}
typedef uint32_t u32x2v __attribute__((ext_vector_type(2)));
__device__ __forceinline__ void buf_store_wt_b64(uint64_t v, __amdgpu_buffer_rsrc_t r, int off) {
  __builtin_amdgcn_raw_buffer_store_b64(u32x2v{uint32_t(v), uint32_t(v >> 32)}, r, off, 0, kWriteThrough);
}

// Transposing sum over the eight lanes u, u + 8, ..., u + 56 of a wave (the
// lanes with equal lane & 7): each of them holds eight values v[0..7], and
// lane 8k + u ends with the total of value k over the eight.  Three butterfly
// steps, each halving the values a lane keeps: partner lane +-8 (DPP row
// rotation by 8), +-16 (permlane16 swap), +-32 (permlane32 swap); at each the
// lane keeps the half its own index bit selects and adds the partner's copy
// of it.  About 24 instructions instead of three reductions per value.
__device__ __forceinline__ float lane_transpose_sum8(const float (&v)[8]) {
  const int lane = __lane_id();
  const bool b0 = (lane >> 3) & 1;
  // step 1: keep the values of index parity b0 (m -> index 2m + b0)
  float w[4];
#pragma unroll
  for (int m = 0; m < 4; ++m) {
    const float keep = b0 ? v[2 * m + 1] : v[2 * m];
    const float send = b0 ? v[2 * m] : v[2 * m + 1];
    w[m] = keep + __uint_as_float(__builtin_amdgcn_update_dpp(0u, __float_as_uint(send), 0x128, 0xF, 0xF, false));
  }
  // step 2: rows 2r and 2r + 1 (lane bit 4); even rows keep m = 0, 2, odd rows m = 1, 3
  float x[2];
#pragma unroll
  for (int n = 0; n < 2; ++n) {
    const auto s = __builtin_amdgcn_permlane16_swap(__float_as_uint(w[2 * n]), __float_as_uint(w[2 * n + 1]), false,
                                                    false);
    x[n] = __uint_as_float(s[0]) + __uint_as_float(s[1]);
  }
  // step 3: lower and upper 32 lanes (lane bit 5); the lower keep n = 0, the upper n = 1
  const auto s = __builtin_amdgcn_permlane32_swap(__float_as_uint(x[0]), __float_as_uint(x[1]), false, false);
  return __uint_as_float(s[0]) + __uint_as_float(s[1]);
}

// Sum over the four 16-lane rows of a wave, every lane getting the total of
// its column (lane & 15): ((row0 + row1) + (row2 + row3)).  gfx950's lane
// swaps do it in the vector ALU, without the LDS crossbar.
__device__ __forceinline__ float row_sum4(float v) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = __uint_as_float(a[0]) + __uint_as_float(a[1]);  // rows (0+1, 0+1, 2+3, 2+3)
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

// Workgroup barrier that orders LDS only.  __syncthreads() also waits for
// every outstanding global load and store of the wave (vmcnt(0)); this one
// leaves them in flight, which a streaming kernel needs to keep its prefetch
// ring going across the barrier.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Sum over the 16 lanes of each row of a wave (every lane gets its row's
// total), in a fixed order, by DPP: quad swaps, then the two row mirrors.
__device__ __forceinline__ float row_sum16(float v) {
  v += __uint_as_float(__builtin_amdgcn_update_dpp(0, __float_as_uint(v), 0xB1, 0xF, 0xF, false));   // lane ^ 1
  v += __uint_as_float(__builtin_amdgcn_update_dpp(0, __float_as_uint(v), 0x4E, 0xF, 0xF, false));   // lane ^ 2
  v += __uint_as_float(__builtin_amdgcn_update_dpp(0, __float_as_uint(v), 0x141, 0xF, 0xF, false));  // 7 - i in 8
  v += __uint_as_float(__builtin_amdgcn_update_dpp(0, __float_as_uint(v), 0x140, 0xF, 0xF, false));  // 15 - i in 16
  return v;
}

// Selection key of token n with score a: larger a ranks first, then the
// smaller index, so distinct tokens never tie.  The score maps onto the upper
// 32 bits order-preservingly, the complemented index onto the lower 12 bits
// (n < 4096).
__device__ __forceinline__ uint32_t order_key(float a) {
  const uint32_t u = __float_as_uint(a);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float order_value(uint32_t k) {
  return __uint_as_float((k & 0x80000000u) ? (k & 0x7fffffffu) : ~k);
}
__device__ __forceinline__ uint64_t sel_key(float a, int n) {
  return (uint64_t(order_key(a)) << 12) | uint64_t(kTokMax - 1 - n);
}

}  // namespace wz

namespace wz {

// Extremes over the 64 lanes of a wave (every lane gets the result), by DPP
// within each 16-lane row and gfx950's lane swaps across rows: no LDS.
template <typename Op>
__device__ __forceinline__ float wave_reduce_f32(float v, Op op) {
  auto dpp = [](float x, auto ctrl) {
    return __uint_as_float(__builtin_amdgcn_update_dpp(0u, __float_as_uint(x), decltype(ctrl)::value, 0xF, 0xF, false));
  };
  v = op(v, dpp(v, std::integral_constant<int, 0xB1>{}));   // lane ^ 1
  v = op(v, dpp(v, std::integral_constant<int, 0x4E>{}));   // lane ^ 2
  v = op(v, dpp(v, std::integral_constant<int, 0x141>{}));  // 7 - i in 8
  v = op(v, dpp(v, std::integral_constant<int, 0x140>{}));  // 15 - i in 16
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = op(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return op(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
__device__ __forceinline__ float wave_min_f32(float v) {
  return wave_reduce_f32(v, [](float a, float b) { return fminf(a, b); });
}
__device__ __forceinline__ float wave_max_f32(float v) {
  return wave_reduce_f32(v, [](float a, float b) { return fmaxf(a, b); });
}

// DPP controls and fp64 / int helpers over a wave's lanes.
constexpr int kDppXor1 = 0xB1;        // quad_perm [1,0,3,2]
constexpr int kDppXor2 = 0x4E;        // quad_perm [2,3,0,1]
constexpr int kDppHalfMirror = 0x141;  // lane i <-> 7 - i within each half row
constexpr int kDppMirror = 0x140;      // lane i <-> 15 - i within each row

template <int CTRL>
__device__ __forceinline__ double dpp_f64(double v) {
  const uint64_t u = __builtin_bit_cast(uint64_t, v);
  const uint32_t lo = uint32_t(__builtin_amdgcn_update_dpp(0, int(uint32_t(u)), CTRL, 0xF, 0xF, false));
  const uint32_t hi = uint32_t(__builtin_amdgcn_update_dpp(0, int(uint32_t(u >> 32)), CTRL, 0xF, 0xF, false));
  return __builtin_bit_cast(double, (uint64_t(hi) << 32) | lo);
}
template <int CTRL>
__device__ __forceinline__ int dpp_i32(int v) {
  return __builtin_amdgcn_update_dpp(0, v, CTRL, 0xF, 0xF, false);
}
__device__ __forceinline__ double readlane_f64(double v, int l) {
  const uint64_t u = __builtin_bit_cast(uint64_t, v);
  const uint32_t lo = uint32_t(__builtin_amdgcn_readlane(int(uint32_t(u)), l));
  const uint32_t hi = uint32_t(__builtin_amdgcn_readlane(int(uint32_t(u >> 32)), l));
  return __builtin_bit_cast(double, (uint64_t(hi) << 32) | lo);
}
__device__ __forceinline__ double permute_f64(int dst_lane, double v) {  // value of lane l goes to lane dst(l)
  const uint64_t u = __builtin_bit_cast(uint64_t, v);
  const uint32_t lo = uint32_t(__builtin_amdgcn_ds_permute(dst_lane * 4, int(uint32_t(u))));
  const uint32_t hi = uint32_t(__builtin_amdgcn_ds_permute(dst_lane * 4, int(uint32_t(u >> 32))));
  return __builtin_bit_cast(double, (uint64_t(hi) << 32) | lo);
}

// op over all 64 lanes (every lane gets the result): within each row of 16
// lanes by DPP, then the four row results in a fixed order.
template <typename Op>
__device__ __forceinline__ double wave_reduce_f64(double v, Op op) {
  v = op(v, dpp_f64<kDppXor1>(v));
  v = op(v, dpp_f64<kDppXor2>(v));
  v = op(v, dpp_f64<kDppHalfMirror>(v));
  v = op(v, dpp_f64<kDppMirror>(v));
  return op(op(readlane_f64(v, 0), readlane_f64(v, 16)), op(readlane_f64(v, 32), readlane_f64(v, 48)));
}
template <typename Op>
__device__ __forceinline__ uint64_t wave_reduce_u64(uint64_t v, Op op) {
  auto dpp = [](uint64_t x, auto ctrl) {
    constexpr int c = decltype(ctrl)::value;
    const uint32_t lo = uint32_t(__builtin_amdgcn_update_dpp(0, int(uint32_t(x)), c, 0xF, 0xF, false));
    const uint32_t hi = uint32_t(__builtin_amdgcn_update_dpp(0, int(uint32_t(x >> 32)), c, 0xF, 0xF, false));
    return (uint64_t(hi) << 32) | lo;
  };
  auto rl = [](uint64_t x, int l) {
    return (uint64_t(uint32_t(__builtin_amdgcn_readlane(int(uint32_t(x >> 32)), l))) << 32) |
           uint32_t(__builtin_amdgcn_readlane(int(uint32_t(x)), l));
  };
  v = op(v, dpp(v, std::integral_constant<int, kDppXor1>{}));
  v = op(v, dpp(v, std::integral_constant<int, kDppXor2>{}));
  v = op(v, dpp(v, std::integral_constant<int, kDppHalfMirror>{}));
  v = op(v, dpp(v, std::integral_constant<int, kDppMirror>{}));
  return op(op(rl(v, 0), rl(v, 16)), op(rl(v, 32), rl(v, 48)));
}
__device__ __forceinline__ int wave_reduce_sum_i32(int v) {
  v += dpp_i32<kDppXor1>(v);
  v += dpp_i32<kDppXor2>(v);
  v += dpp_i32<kDppHalfMirror>(v);
  v += dpp_i32<kDppMirror>(v);
  return (__builtin_amdgcn_readlane(v, 0) + __builtin_amdgcn_readlane(v, 16)) +
         (__builtin_amdgcn_readlane(v, 32) + __builtin_amdgcn_readlane(v, 48));
}

// Inclusive prefix sum over the 64 lanes of a wave: shifts within each
// 16-lane row by DPP, then the totals of the rows below from three lane reads.
__device__ __forceinline__ int wave_incl_scan_i32(int v) {
  v += __builtin_amdgcn_update_dpp(0, v, 0x111, 0xF, 0xF, false);  // row_shr:1
  v += __builtin_amdgcn_update_dpp(0, v, 0x112, 0xF, 0xF, false);  // row_shr:2
  v += __builtin_amdgcn_update_dpp(0, v, 0x114, 0xF, 0xF, false);  // row_shr:4
  v += __builtin_amdgcn_update_dpp(0, v, 0x118, 0xF, 0xF, false);  // row_shr:8
  const int r0 = __builtin_amdgcn_readlane(v, 15), r1 = __builtin_amdgcn_readlane(v, 31),
            r2 = __builtin_amdgcn_readlane(v, 47);
  const int row = (threadIdx.x & 63) >> 4;
  return v + (row > 0 ? r0 : 0) + (row > 1 ? r1 : 0) + (row > 2 ? r2 : 0);
}

}  // namespace wz
