// Shared device helpers of the LiLiCorr HIP library (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "lilicorr.h"

namespace lilicorr {

constexpr int kWave = 64;

// ---- status helpers (host) --------------------------------------------------------------------
inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

inline lilicorr_status launch_status() {
  return hipGetLastError() == hipSuccess ? LILICORR_OK : LILICORR_ERR_HIP;
}

// ---- wave primitives --------------------------------------------------------------------------
__device__ __forceinline__ int lane_id() { return __lane_id(); }

__device__ __forceinline__ uint32_t readlane32(uint32_t v, int lane) {
  return (uint32_t)__builtin_amdgcn_readlane((int)v, lane);
}

__device__ __forceinline__ uint64_t readlane64(uint64_t v, int lane) {
  uint32_t lo = readlane32((uint32_t)v, lane);
  uint32_t hi = readlane32((uint32_t)(v >> 32), lane);
  return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ float readlanef(float v, int lane) {
  return __uint_as_float(readlane32(__float_as_uint(v), lane));
}

__device__ __forceinline__ uint32_t uniform32(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_readfirstlane((int)v);
}

__device__ __forceinline__ uint64_t uniform64(uint64_t v) {
  return ((uint64_t)uniform32((uint32_t)(v >> 32)) << 32) | uniform32((uint32_t)v);
}

// lane l receives v from lane l-1 (DPP wave_shr:1); lane 0 receives 0
__device__ __forceinline__ uint64_t shift_up64(uint64_t v) {
  uint32_t lo = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)v, 0x138, 0xf, 0xf, false);
  uint32_t hi = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)(v >> 32), 0x138, 0xf, 0xf, false);
  return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ uint64_t shfl_xor64(uint64_t v, int mask) {
  uint32_t lo = (uint32_t)__shfl_xor((int)(uint32_t)v, mask, kWave);
  uint32_t hi = (uint32_t)__shfl_xor((int)(uint32_t)(v >> 32), mask, kWave);
  return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ uint64_t shfl64(uint64_t v, int src) {
  uint32_t lo = (uint32_t)__shfl((int)(uint32_t)v, src, kWave);
  uint32_t hi = (uint32_t)__shfl((int)(uint32_t)(v >> 32), src, kWave);
  return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, kWave);
  return v;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v = fmaxf(v, __shfl_xor(v, m, kWave));
  return v;
}

// ---- candidate keys ---------------------------------------------------------------------------
// A candidate (value x, token id) is ranked by x descending, then id ascending. The 64-bit key
//   (order(x) << 32) | (0xFFFFFFFF - id)
// is larger for the better candidate; order() maps floats monotonically to unsigned integers and
// folds -0 onto +0. The key 0 is below every real key and marks an empty list slot.
__device__ __forceinline__ uint32_t order_bits(float x) {
  uint32_t b = __float_as_uint(x);
  if (b == 0x80000000u) b = 0u;
  return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

__device__ __forceinline__ float order_value(uint32_t k) {
  return __uint_as_float((k & 0x80000000u) ? (k & 0x7fffffffu) : ~k);
}

__device__ __forceinline__ uint64_t make_key(float x, uint32_t id) {
  return ((uint64_t)order_bits(x) << 32) | (uint64_t)(0xFFFFFFFFu - id);
}

__device__ __forceinline__ float key_value(uint64_t key) {
  return key == 0 ? -__builtin_inff() : order_value((uint32_t)(key >> 32));
}

__device__ __forceinline__ uint32_t key_id(uint64_t key) { return 0xFFFFFFFFu - (uint32_t)key; }

// Top-64 of the union of two lists that are each sorted descending across the 64 lanes
// (bitonic merge: the lane-wise max of a and reversed b is bitonic, then 6 half-cleaners).
__device__ __forceinline__ uint64_t merge_desc64(uint64_t a, uint64_t b) {
  const int lane = lane_id();
  uint64_t br = shfl64(b, kWave - 1 - lane);
  uint64_t c = a > br ? a : br;
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) {
    uint64_t o = shfl_xor64(c, m);
    bool lower = (lane & m) == 0;
    c = lower ? (c > o ? c : o) : (c < o ? c : o);
  }
  return c;
}

// Full descending bitonic sort of one float per lane.
__device__ __forceinline__ float sort_desc64(float v) {
  const int lane = lane_id();
#pragma unroll
  for (int k = 2; k <= kWave; k <<= 1) {
#pragma unroll
    for (int j = k >> 1; j >= 1; j >>= 1) {
      float o = __shfl_xor(v, j, kWave);
      bool keep_max = ((lane & j) == 0) == ((lane & k) == 0);
      v = keep_max ? fmaxf(v, o) : fminf(v, o);
    }
  }
  return v;
}

}  // namespace lilicorr
