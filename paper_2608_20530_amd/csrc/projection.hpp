// Device helpers of the candidate projection u = E[id] W on the bf16 matrix cores, shared by the
// candidate-vector kernel and the fused scoring kernel.
//
// Every fp32 weight is split exactly into three bf16 terms (hi + mid + lo == w); E is bf16, so each
// bf16 x bf16 product is exact in fp32 and fp32 accumulation gives fp32-grade results.
//
// Packed weight layout (written by lilicorr_pack_weights):
//   [side 2][k-block dkp][term 3][column block nbp][lane 64][8 bf16]: v_mfma_f32_16x16x32_bf16
//     B fragments; lane l of block (kb, nb) holds W[kb*32 + (l/16)*8 + i][nb*16 + l%16], i = 0..7
//     (0 for rows or columns at or beyond d)
//   followed by [side 2][d][d] fp32 copies (used by the fp32-embedding kernel)
// Side 0 is W_in, side 1 is W_out. nbp is d/16 rounded up to whole wave column groups and dkp is
// the number of 32-deep k-blocks rounded up to even, so the MFMA loop never branches.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "common.hpp"

namespace lilicorr {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// The packed layout pads the output columns to whole groups of kNbPerWave 16-column blocks (the
// candidate-vector kernel's waves own one group each); a kernel may give its waves fewer blocks
// (NB, a divisor of kNbPerWave) and so run more waves over the same layout.
constexpr int kNbPerWave = 4;

struct VecGeom {
  int d16;    // 16-column blocks of the output
  int nbp;    // d16 rounded up to whole waves (kNbPerWave blocks each)
  int dk;     // 32-deep k-blocks of the contraction
  int dkp;    // dk rounded up to even (the MFMA loop handles two k-blocks per trip)
  int waves;  // waves per side: one per kNbPerWave column blocks
  int rm;     // 16-row blocks per workgroup of the candidate-vector kernel
};

// rm: 64-row tiles up to d = 512 (two workgroups per compute unit; at d <= 256 a 128-row tile's
// 8 x 4 accumulator blocks plus two weight buffers exceed the 256 registers of two waves per
// SIMD and spilled: 175 against 160 us at 131072 rows, d = 256; at 256 < d <= 512 it needs 133 KB
// of LDS, one workgroup per compute unit, and measured 7% slower at 131072 rows, d = 512);
// 32-row tiles above d = 512. (Many tiles at 448 < d <= 512 take the persistent kernels.)
inline VecGeom vec_geom(int d, int64_t M = 0) {
  VecGeom g;
  g.d16 = d / 16;
  g.nbp = (g.d16 + kNbPerWave - 1) / kNbPerWave * kNbPerWave;
  g.dk = (d + 31) / 32;
  g.dkp = (g.dk + 1) / 2 * 2;
  g.waves = g.nbp / kNbPerWave;
  (void)M;
  g.rm = d > 512 ? 2 : 4;
  return g;
}

inline size_t frag_bytes(int d) {
  VecGeom g = vec_geom(d);
  return (size_t)2 * g.dkp * 3 * g.nbp * 1024;
}

inline size_t packed_bytes(int d) { return frag_bytes(d) + (size_t)2 * d * d * sizeof(float); }

template <int NB = kNbPerWave>
using BFrag = u32x4[NB][3];

// B fragments of k-block kb for a wave's NB column blocks, three terms each; wf points at the
// wave's first column block (plus lane * 16) in k-block 0, term 0 of its side
template <int NB>
__device__ __forceinline__ void load_bfrag(BFrag<NB>& dst, const unsigned char* wf, size_t slice,
                                           int kb) {
  const unsigned char* p = wf + (size_t)kb * 3 * slice;
#pragma unroll
  for (int t = 0; t < 3; ++t)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
      dst[nb][t] = *reinterpret_cast<const u32x4*>(p + t * slice + nb * 1024);
}

// acc[mb][nb] += A[rows of block mb][k-block kb] x B[k-block kb][column block nb], all three
// terms; the term loop is outermost so consecutive MFMAs never feed each other
template <int RM, int NB>
__device__ __forceinline__ void mfma_kblock(f32x4 (&acc)[RM][NB], const BFrag<NB>& b,
                                            const uint16_t* A, int astride, int kb, int lane) {
  bf16x8 a[RM];
  const int kcol = kb * 32 + (lane >> 4) * 8;
#pragma unroll
  for (int mb = 0; mb < RM; ++mb)
    a[mb] = __builtin_bit_cast(
        bf16x8, *reinterpret_cast<const u32x4*>(A + (mb * 16 + (lane & 15)) * astride + kcol));
#pragma unroll
  for (int t = 0; t < 3; ++t)
#pragma unroll
    for (int mb = 0; mb < RM; ++mb)
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
        acc[mb][nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
            a[mb], __builtin_bit_cast(bf16x8, b[nb][t]), acc[mb][nb], 0, 0, 0);
}

// The whole contraction of a wave's RM row blocks x NB column blocks. b0 must already hold
// k-block 0 (so its loads can overlap whatever precedes). Two k-blocks per trip through two
// register buffers: the loads of the next k-block are in flight while the MFMAs of the current
// one run (the last trip reloads the final k-block instead of reading past the weights).
template <int RM, int NB>
__device__ __forceinline__ void project_tile(f32x4 (&acc)[RM][NB], BFrag<NB>& b0,
                                             const uint16_t* A, int astride,
                                             const unsigned char* wf, size_t slice, int dkp,
                                             int lane) {
#pragma unroll
  for (int mb = 0; mb < RM; ++mb)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) acc[mb][nb] = f32x4{0.f, 0.f, 0.f, 0.f};
  BFrag<NB> b1;
  // the scheduling barriers keep each k-block's twelve fragment loads issued together ahead of
  // the MFMAs of the previous one: left alone, the scheduler interleaves them into the MFMA
  // stream to save registers and then waits on loads it has just issued
  for (int kb = 0; kb < dkp; kb += 2) {
    load_bfrag(b1, wf, slice, kb + 1);
    __builtin_amdgcn_sched_barrier(0);
    mfma_kblock<RM, NB>(acc, b0, A, astride, kb, lane);
    __builtin_amdgcn_sched_barrier(0);
    load_bfrag(b0, wf, slice, kb + 2 < dkp ? kb + 2 : dkp - 1);
    __builtin_amdgcn_sched_barrier(0);
    mfma_kblock<RM, NB>(acc, b1, A, astride, kb + 1, lane);
    __builtin_amdgcn_sched_barrier(0);
  }
}

// The same contraction with the weight fragments one column block at a time through four
// register buffers (three in flight): 48 registers of weights instead of 96, for a kernel held to
// 128 registers (1024-thread workgroups). Buffer p % 4 of piece p = (k-block, column block) is the
// column block itself, so the ring index is fixed at compile time; each accumulator sees the same
// sequence of MFMAs as in project_tile, so the results are identical.
template <int RM>
__device__ __forceinline__ void project_tile_lean(f32x4 (&acc)[RM][kNbPerWave], const uint16_t* A,
                                                  int astride, const unsigned char* wf,
                                                  size_t slice, int dkp, int lane) {
  constexpr int NB = kNbPerWave;
  static_assert(NB == 4, "one register buffer per column block");
#pragma unroll
  for (int mb = 0; mb < RM; ++mb)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) acc[mb][nb] = f32x4{0.f, 0.f, 0.f, 0.f};
  u32x4 bq[NB][3];
  auto load = [&](int kb, int nb) {
    const unsigned char* q = wf + (size_t)kb * 3 * slice + nb * 1024;
#pragma unroll
    for (int t = 0; t < 3; ++t) bq[nb][t] = *reinterpret_cast<const u32x4*>(q + t * slice);
  };
  load(0, 0);
  load(0, 1);
  load(0, 2);
  for (int kb = 0; kb < dkp; ++kb) {
    bf16x8 a[RM];
    const int kcol = kb * 32 + (lane >> 4) * 8;
#pragma unroll
    for (int mb = 0; mb < RM; ++mb)
      a[mb] = __builtin_bit_cast(
          bf16x8, *reinterpret_cast<const u32x4*>(A + (mb * 16 + (lane & 15)) * astride + kcol));
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      // piece 4 kb + nb + 3: column block nb + 3 of this k-block, or nb - 1 of the next
      if (nb == 0) load(kb, 3);
      else if (kb + 1 < dkp) load(kb + 1, nb - 1);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int t = 0; t < 3; ++t)
#pragma unroll
        for (int mb = 0; mb < RM; ++mb)
          acc[mb][nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
              a[mb], __builtin_bit_cast(bf16x8, bq[nb][t]), acc[mb][nb], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
  }
}

// Gather `rows` embedding rows into the bf16 A tile (row stride astride, dpad columns, zero past
// d). rid[r] must hold the row's token id, or -1 for a zero row (ids outside [0, V) were already
// mapped to -1). Eight independent 16-byte loads in flight per thread.
__device__ __forceinline__ void gather_rows(uint16_t* A, int astride, int rows,
                                            const int32_t* rid, const uint16_t* E, int d,
                                            int dpad, int tid, int nthreads) {
  const int cpr = dpad / 8;  // 16-byte chunks per LDS row
  for (int i0 = tid; i0 < rows * cpr; i0 += 8 * nthreads) {
    u32x4 v[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const int i = i0 + q * nthreads;
      v[q] = u32x4{0u, 0u, 0u, 0u};
      if (i < rows * cpr) {
        const int r = i / cpr, c = i - r * cpr;
        const int32_t id = rid[r];
        if (id >= 0 && c * 8 < d) v[q] = *reinterpret_cast<const u32x4*>(E + (int64_t)id * d + c * 8);
      }
    }
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const int i = i0 + q * nthreads;
      if (i < rows * cpr) {
        const int r = i / cpr, c = i - r * cpr;
        *reinterpret_cast<u32x4*>(A + r * astride + c * 8) = v[q];
      }
    }
  }
}

// Per-wave partial squared norms of the tile's rows: lane l holds rows (l/16)*4 + i of each row
// block and column l%16 of each column block (padding columns hold zeros); ss[row] receives the
// sum over this wave's NB * 16 columns.
template <int RM, int NB>
__device__ __forceinline__ void row_sumsq(const f32x4 (&acc)[RM][NB], float* ss, int lane) {
#pragma unroll
  for (int mb = 0; mb < RM; ++mb) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float s = 0.f;
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) s = fmaf(acc[mb][nb][i], acc[mb][nb][i], s);
      s += __shfl_xor(s, 1, kWave);
      s += __shfl_xor(s, 2, kWave);
      s += __shfl_xor(s, 4, kWave);
      s += __shfl_xor(s, 8, kWave);
      if ((lane & 15) == 0) ss[mb * 16 + (lane >> 4) * 4 + i] = s;
    }
  }
}

}  // namespace lilicorr
