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

// Wave-wide reductions on DPP (row shifts within 16-lane rows, then row broadcasts); the result
// lands in lane 63 and is read back as a wave-uniform value. Lanes a DPP step cannot source
// receive the identity.
template <int CTRL, int ROW_MASK, int BANK_MASK>
__device__ __forceinline__ float dpp_f32(float identity, float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(identity), __float_as_int(x),
                                                    CTRL, ROW_MASK, BANK_MASK, false));
}

template <typename Op>
__device__ __forceinline__ float wave_reduce_dpp(float v, float identity, Op op) {
  // after the row shifts by 1, 2, 4, 8 lane 15 of each 16-lane row holds that row's total
  v = op(v, dpp_f32<0x111, 0xf, 0xf>(identity, v));  // row_shr:1
  v = op(v, dpp_f32<0x112, 0xf, 0xf>(identity, v));  // row_shr:2
  v = op(v, dpp_f32<0x114, 0xf, 0xf>(identity, v));  // row_shr:4
  v = op(v, dpp_f32<0x118, 0xf, 0xf>(identity, v));  // row_shr:8
  v = op(v, dpp_f32<0x142, 0xa, 0xf>(identity, v));  // row_bcast:15 into rows 1 and 3
  v = op(v, dpp_f32<0x143, 0xc, 0xf>(identity, v));  // row_bcast:31 into rows 2 and 3
  return readlanef(v, 63);
}

__device__ __forceinline__ float wave_max_dpp(float v) {
  return wave_reduce_dpp(v, -__builtin_inff(), [](float a, float b) { return fmaxf(a, b); });
}

__device__ __forceinline__ float wave_sum_dpp(float v) {
  return wave_reduce_dpp(v, 0.f, [](float a, float b) { return a + b; });
}

// ---- staging global memory into LDS ------------------------------------------------------------
// Every thread issues up to BATCH independent loads before its first LDS store, so a staging pass
// costs one memory round trip per batch instead of one per element.
typedef unsigned int stage_u32x4 __attribute__((ext_vector_type(4)));

template <int BATCH, typename T>
__device__ __forceinline__ void stage_to_lds(T* __restrict__ dst, const T* __restrict__ src,
                                             int64_t n, int tid, int nthreads) {
  for (int64_t base = tid; base < n; base += (int64_t)BATCH * nthreads) {
    T v[BATCH];
#pragma unroll
    for (int b = 0; b < BATCH; ++b) {
      const int64_t i = base + (int64_t)b * nthreads;
      if (i < n) v[b] = src[i];
    }
#pragma unroll
    for (int b = 0; b < BATCH; ++b) {
      const int64_t i = base + (int64_t)b * nthreads;
      if (i < n) dst[i] = v[b];
    }
  }
}

// As stage_to_lds for 4-byte words, moving 16-byte chunks when both addresses allow it.
__device__ __forceinline__ void stage_words(void* dst, const void* src, int64_t nwords, int tid,
                                            int nthreads) {
  if (((reinterpret_cast<uintptr_t>(src) | reinterpret_cast<uintptr_t>(dst)) & 15u) == 0) {
    const int64_t n16 = nwords / 4;
    stage_to_lds<8>(static_cast<stage_u32x4*>(dst), static_cast<const stage_u32x4*>(src), n16, tid,
                    nthreads);
    const int64_t done = n16 * 4;
    if (tid < nwords - done)
      static_cast<uint32_t*>(dst)[done + tid] = static_cast<const uint32_t*>(src)[done + tid];
  } else {
    stage_to_lds<8>(static_cast<uint32_t*>(dst), static_cast<const uint32_t*>(src), nwords, tid,
                    nthreads);
  }
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

// Full descending bitonic sort of one 64-bit key per lane.
__device__ __forceinline__ uint64_t sort_desc64_u64(uint64_t v) {
  const int lane = lane_id();
#pragma unroll
  for (int k = 2; k <= kWave; k <<= 1) {
#pragma unroll
    for (int j = k >> 1; j >= 1; j >>= 1) {
      const uint64_t o = shfl_xor64(v, j);
      const bool keep_max = ((lane & j) == 0) == ((lane & k) == 0);
      v = keep_max ? (v > o ? v : o) : (v < o ? v : o);
    }
  }
  return v;
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

// ---- one row of the walk -----------------------------------------------------------------------
// all-reduce over aligned groups of G lanes; every lane of a group receives the group's result
template <typename Op>
__device__ __forceinline__ float dpp_allreduce16(float v, Op op) {
  v = op(v, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0xB1, 0xf, 0xf, false)));   // quad_perm 1,0,3,2
  v = op(v, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x4E, 0xf, 0xf, false)));   // quad_perm 2,3,0,1
  v = op(v, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x141, 0xf, 0xf, false)));  // row_half_mirror
  v = op(v, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x140, 0xf, 0xf, false)));  // row_mirror
  return v;
}

template <int G, typename Op>
__device__ __forceinline__ float group_allreduce(float v, Op op) {
  v = dpp_allreduce16(v, op);
  if (G >= 32) v = op(v, __shfl_xor(v, 16, kWave));
  if (G >= 64) v = op(v, __shfl_xor(v, 32, kWave));
  return v;
}

// One row of the walk's transition table, resolved by an aligned group of G lanes (lane j of the
// group holds z_j; lanes with live == false hold no candidate): the lowest j attaining max z
// (0 if none does, which only NaN scores cause) and the local log-likelihood
// -log sum_j exp(z_j - max z) of Eq. (localar), both in fp32. Every lane of the wave must call it.
// m receives the row's maximum.
template <int G>
__device__ __forceinline__ void resolve_row(float z, bool live, int& arg, float& lq, float& m) {
  const int gshift = (lane_id() / G) * G;  // first ballot bit of this lane's group
  const uint64_t gmask = G == 64 ? ~0ull : ((1ull << G) - 1);
  m = group_allreduce<G>(live ? z : -__builtin_inff(),
                         [](float a, float b) { return fmaxf(a, b); });
  const uint64_t hits = (__ballot(live && z == m) >> gshift) & gmask;
  arg = hits ? __ffsll((long long)hits) - 1 : 0;
  const float s = group_allreduce<G>(live ? expf(z - m) : 0.f,
                                     [](float a, float b) { return a + b; });
  lq = -logf(s);
}

template <int G>
__device__ __forceinline__ void resolve_row(float z, bool live, int& arg, float& lq) {
  float m;
  resolve_row<G>(z, live, arg, lq, m);
}

// table entry: low 32 bits the argmax, high 32 bits the fp32 local log-likelihood
__device__ __forceinline__ uint64_t table_entry(int arg, float lq) {
  return (uint64_t)(uint32_t)arg | ((uint64_t)__float_as_uint(lq) << 32);
}

}  // namespace lilicorr
