// Wave-wide inclusive scans over the 64 lanes of a wavefront with DPP
// moves (shared by the planner and the one-launch lookup kernels).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace dpi {
namespace {

template <int CTRL>
__device__ __forceinline__ int64_t dpp_move(int64_t x) {
  const int lo = __builtin_amdgcn_mov_dpp((int)(uint32_t)(uint64_t)x, CTRL, 0xf, 0xf, false);
  const int hi = __builtin_amdgcn_mov_dpp((int)(uint32_t)((uint64_t)x >> 32), CTRL, 0xf, 0xf, false);
  return (int64_t)(((uint64_t)(uint32_t)hi << 32) | (uint64_t)(uint32_t)lo);
}

// Inclusive scan over the 64 lanes: shifts within rows of 16 lanes, then the
// row-15 and lane-31 broadcasts.  Lanes whose DPP source does not exist never
// add what they received.
__device__ __forceinline__ int64_t wave_incl_scan(int64_t x, int lane) {
  const int r = lane & 15;
  int64_t y;
  y = dpp_move<0x111>(x);   // row_shr:1
  x = r >= 1 ? x + y : x;
  y = dpp_move<0x112>(x);   // row_shr:2
  x = r >= 2 ? x + y : x;
  y = dpp_move<0x114>(x);   // row_shr:4
  x = r >= 4 ? x + y : x;
  y = dpp_move<0x118>(x);   // row_shr:8
  x = r >= 8 ? x + y : x;
  y = dpp_move<0x142>(x);   // row_bcast:15
  x = (lane & 16) ? x + y : x;
  y = dpp_move<0x143>(x);   // row_bcast:31
  x = lane >= 32 ? x + y : x;
  return x;
}

template <int CTRL>
__device__ __forceinline__ uint32_t dpp_move_u32(uint32_t x) {
  return (uint32_t)__builtin_amdgcn_mov_dpp((int)x, CTRL, 0xf, 0xf, false);
}

// The same scan for values whose wave total fits 32 bits.
__device__ __forceinline__ uint32_t wave_incl_scan32(uint32_t x, int lane) {
  const int r = lane & 15;
  uint32_t y;
  y = dpp_move_u32<0x111>(x);
  x = r >= 1 ? x + y : x;
  y = dpp_move_u32<0x112>(x);
  x = r >= 2 ? x + y : x;
  y = dpp_move_u32<0x114>(x);
  x = r >= 4 ? x + y : x;
  y = dpp_move_u32<0x118>(x);
  x = r >= 8 ? x + y : x;
  y = dpp_move_u32<0x142>(x);
  x = (lane & 16) ? x + y : x;
  y = dpp_move_u32<0x143>(x);
  x = lane >= 32 ? x + y : x;
  return x;
}

// Lane l's 64-bit value, read by every lane (l wave-uniform).
__device__ __forceinline__ int64_t lane_value(int64_t x, int l) {
  const uint32_t lo = __builtin_amdgcn_readlane((uint32_t)(uint64_t)x, l);
  const uint32_t hi = __builtin_amdgcn_readlane((uint32_t)((uint64_t)x >> 32), l);
  return (int64_t)(((uint64_t)hi << 32) | lo);
}

}  // namespace
}  // namespace dpi
