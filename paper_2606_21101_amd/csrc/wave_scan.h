// Wave-wide inclusive scans over the 64 lanes of a wavefront with DPP
// moves (shared by the planner and the one-launch lookup kernels).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace dpi {
namespace {

// DPP move in which lanes whose source lies outside the pattern, and lanes of
// rows outside ROWS (a row mask), receive 0: each scan step is then one
// unconditional add.
template <int CTRL, int ROWS>
__device__ __forceinline__ uint32_t dpp_or_zero(uint32_t x) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, CTRL, ROWS, 0xf, true);
}

typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

template <int CTRL, int ROWS>
__device__ __forceinline__ int64_t dpp_or_zero(int64_t x) {
  const u32x2 v = __builtin_bit_cast(u32x2, x);
  // the halves moved into one register pair: one 64-bit add per step
  return __builtin_bit_cast(int64_t, u32x2{dpp_or_zero<CTRL, ROWS>(v.x), dpp_or_zero<CTRL, ROWS>(v.y)});
}

// Inclusive scan over the 64 lanes: shifts by 1, 2, 4 and 8 within rows of
// 16 lanes, then row 0's total into row 1 and row 2's into row 3 (row_bcast
// 15), then rows 0-1's total into rows 2 and 3 (row_bcast 31).
template <typename X>
__device__ __forceinline__ X wave_incl_scan_t(X x) {
  x += dpp_or_zero<0x111, 0xf>(x);   // row_shr:1
  x += dpp_or_zero<0x112, 0xf>(x);   // row_shr:2
  x += dpp_or_zero<0x114, 0xf>(x);   // row_shr:4
  x += dpp_or_zero<0x118, 0xf>(x);   // row_shr:8
  x += dpp_or_zero<0x142, 0xa>(x);   // row_bcast:15, rows 1 and 3
  x += dpp_or_zero<0x143, 0xc>(x);   // row_bcast:31, rows 2 and 3
  return x;
}

__device__ __forceinline__ int64_t wave_incl_scan(int64_t x, int lane) {
  (void)lane;
  return wave_incl_scan_t<int64_t>(x);
}

// The same scan for values whose wave total fits 32 bits.
__device__ __forceinline__ uint32_t wave_incl_scan32(uint32_t x, int lane) {
  (void)lane;
  return wave_incl_scan_t<uint32_t>(x);
}

// Lane l's 64-bit value, read by every lane (l wave-uniform).
__device__ __forceinline__ int64_t lane_value(int64_t x, int l) {
  const uint32_t lo = __builtin_amdgcn_readlane((uint32_t)(uint64_t)x, l);
  const uint32_t hi = __builtin_amdgcn_readlane((uint32_t)((uint64_t)x >> 32), l);
  return (int64_t)(((uint64_t)hi << 32) | lo);
}

}  // namespace
}  // namespace dpi
