// The exact max-path decode of one request by one workgroup (decode-rule appendix, Eq. pathscore),
// shared by the stand-alone decode kernel and the fused scoring kernel.
//
// g(c) = P_0[c_0] + sum_{t>=1} S[t-1][c_{t-1}][c_t] (+ lambda sum_t logp[t][c_t]), P_0 = S0 or all
// zero. Wave 0 sweeps left to right with lane k holding the best score of a path ending at
// candidate k: at each slot it scans the K predecessors in order (a strict '>' keeps the lowest
// index on ties) and stores each lane's predecessor as a byte. Path sums are double: each fp32
// score is widened exactly and every partial sum is rounded once, in the order of the sum above
// (the lambda term, an exact product of two floats in double, after the slot's matching term), so
// the maximiser is the exact one unless two path sums differ by less than that double rounding.
// One lane picks the best final candidate (lowest index on ties) and traces back; then groups of
// G lanes evaluate Eq. (localar) along the path for all slots in parallel. G >= K is also the
// compile-time bound of the predecessor scan.
#pragma once

#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "common.hpp"

namespace lilicorr {

// Row stride, in floats, of the transposed scores a workgroup stages for the sweep: column p of
// S[t] for candidate k sits at T[(t*K + k) * stride + p], padded with -inf from K up to G; the
// four extra floats spread a wave's 16-byte reads over the LDS banks.
template <int G>
__host__ __device__ constexpr int viterbi_stride() { return G + 4; }

// Stage S[n] ([B-1][K][K], global) transposed and padded into T (LDS); every thread calls it.
template <int G>
__device__ __forceinline__ void stage_transposed(float* T, const float* Sn, int64_t B, int K,
                                                 int tid, int nthreads) {
  constexpr int kStride = viterbi_stride<G>();
  const int64_t n = (B - 1) * (int64_t)K * K;
  for (int64_t base = tid; base < n; base += 8 * (int64_t)nthreads) {
    float v[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const int64_t i = base + q * (int64_t)nthreads;
      v[q] = i < n ? Sn[i] : 0.f;
    }
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const int64_t i = base + q * (int64_t)nthreads;
      if (i < n) {
        const int64_t tp = i / K;            // t * K + p
        const int k = (int)(i - tp * K);
        const int64_t t = tp / K;
        const int p = (int)(tp - t * K);
        T[(t * K + k) * kStride + p] = v[q];
      }
    }
  }
  const int pad = G - K;
  for (int64_t i = tid; i < (B - 1) * (int64_t)K * pad; i += nthreads) {
    const int64_t row = i / pad;
    T[row * kStride + K + (int)(i - row * pad)] = -__builtin_inff();
  }
}

// Every thread of the workgroup calls this (it holds barriers); nthreads is a multiple of 64.
//   STAGED Sv is T, the transposed and padded scores in LDS (stage_transposed); otherwise Sv is
//          S[n] itself, [B-1][K][K] row-major in global memory. Unused when B == 1.
//   S0n    the request's anchor scores [K], or null for all zero
//   lpn    its [B][K] drafter log-probabilities (read only when lambda != 0)
//   idn    its [B][K] candidate ids
//   from   B * K bytes of LDS, path B bytes of LDS, line 64 doubles of LDS (16-byte aligned)
//   draft_n [B]; choice_n [B], logq_n [B], score_n [1] may be null
// The sweep runs in wave 0 alone. Each slot's best path sums are published through `line` (-inf
// for lanes past K) and read back by every lane as 16-byte broadcasts; a wave's LDS operations
// complete in order, so no barrier is needed between that write and the reads. Candidates past K
// score -inf against every predecessor, so the scan needs no test on K.
template <int G, bool STAGED>
__device__ __forceinline__ void viterbi_block(const float* Sv, const float* S0n, const float* lpn,
                                              const int32_t* idn, int64_t B, int K, float lambda,
                                              uint8_t* from, uint8_t* path, double* line,
                                              int32_t* draft_n, int32_t* choice_n, float* logq_n,
                                              float* score_n, int tid, int nthreads) {
  typedef float f4 __attribute__((ext_vector_type(4)));
  typedef double d2 __attribute__((ext_vector_type(2)));
  constexpr int kStride = viterbi_stride<G>();
  const bool use_lp = lambda != 0.f;
  const double lam = (double)lambda;
  if (tid < kWave) {
    const int k = tid;
    const bool live = k < K;
    double best = -__builtin_inf();
    if (live) {
      best = S0n ? (double)S0n[k] : 0.0;
      if (use_lp) best += lam * (double)lpn[k];
    }
    for (int64_t t = 1; t < B; ++t) {
      line[k] = best;
      double bv;
      int bp = 0;
      if (STAGED) {
        // lane k's column of S[t-1] is row (t-1, k) of T; rows of dead lanes are not read
        const float* Tk = Sv + ((t - 1) * K + (live ? k : 0)) * (int64_t)kStride;
        f4 c4[G / 4];
#pragma unroll
        for (int q = 0; q < G / 4; ++q) c4[q] = *reinterpret_cast<const f4*>(Tk + 4 * q);
        bv = line[0] + (double)c4[0][0];
#pragma unroll
        for (int q = 0; q < G / 4; ++q) {
          const d2 b01 = *reinterpret_cast<const d2*>(line + 4 * q);
          const d2 b23 = *reinterpret_cast<const d2*>(line + 4 * q + 2);
#pragma unroll
          for (int e = (q == 0 ? 1 : 0); e < 4; ++e) {
            const double v = (e < 2 ? b01[e & 1] : b23[e & 1]) + (double)c4[q][e];
            if (v > bv) {
              bv = v;
              bp = 4 * q + e;
            }
          }
        }
      } else {
        // lane k's column of S[t-1], loaded 16 predecessors at a time ahead of their scan (one
        // memory latency per 16 predecessors rather than one per predecessor)
        const float* St = Sv + (t - 1) * (int64_t)K * K;
        constexpr int kBatch = 16;
        bv = -__builtin_inf();
#pragma unroll
        for (int p0 = 0; p0 < G; p0 += kBatch) {
          float c[kBatch];
#pragma unroll
          for (int q = 0; q < kBatch; ++q)
            c[q] = live && p0 + q < K ? St[(p0 + q) * K + k] : 0.f;
#pragma unroll
          for (int q = 0; q < kBatch; ++q) {
            const int p = p0 + q;
            if (p < K) {
              const double v = line[p] + (double)c[q];
              if (p == 0 || v > bv) {
                bv = v;
                bp = p;
              }
            }
          }
        }
      }
      if (live) {
        if (use_lp) bv += lam * (double)lpn[t * K + k];
        from[t * K + k] = (uint8_t)bp;
      } else {
        bv = -__builtin_inf();
      }
      best = bv;
    }
    // best final candidate (lowest index on ties), the same scan in every lane
    line[k] = best;
    int c = 0;
    double g = line[0];
#pragma unroll
    for (int q = 0; q < G / 2; ++q) {
      const d2 b2 = *reinterpret_cast<const d2*>(line + 2 * q);
#pragma unroll
      for (int e = (q == 0 ? 1 : 0); e < 2; ++e) {
        if (b2[e] > g) {
          g = b2[e];
          c = 2 * q + e;
        }
      }
    }
    if (k == 0) {
      if (score_n) *score_n = (float)g;
      path[B - 1] = (uint8_t)c;
      for (int64_t t = B - 1; t >= 1; --t) {
        c = from[t * K + c];
        path[t - 1] = (uint8_t)c;
      }
    }
  }
  __syncthreads();

  // logq along the path: row t holds z_t[k] = P_t(c_{t-1}, k) (+ lambda logp[t][k])
  const int j = tid % G;
  const int group = tid / G;
  const int ngroups = nthreads / G;
  const bool live = j < K;
  for (int64_t base = 0; base < B; base += ngroups) {
    const int64_t t = base + group;
    float z = 0.f;
    int ct = 0;
    if (t < B) {
      ct = path[t];
      if (live) {
        if (t == 0)
          z = S0n ? S0n[j] : 0.f;
        else if (STAGED)
          z = Sv[((t - 1) * K + j) * (int64_t)kStride + path[t - 1]];
        else
          z = Sv[((t - 1) * K + path[t - 1]) * (int64_t)K + j];
        if (use_lp) z = fmaf(lambda, lpn[t * K + j], z);
      }
    }
    const float m = group_allreduce<G>(live ? z : -__builtin_inff(),
                                       [](float a, float b) { return fmaxf(a, b); });
    const float s = group_allreduce<G>(live ? expf(z - m) : 0.f,
                                       [](float a, float b) { return a + b; });
    // z at the committed candidate, from its lane of the group
    const float zc = __shfl(z, (tid & (kWave - 1)) - j + ct, kWave);
    if (t < B && j == 0) {
      draft_n[t] = idn[t * K + ct];
      if (choice_n) choice_n[t] = ct;
      if (logq_n) logq_n[t] = (zc - m) - logf(s);
    }
  }
}

}  // namespace lilicorr
