// Certified greedy decisions: a walk decision whose fp32 node scores leave the winner within a
// margin of another candidate is decided again in double precision.
//
// The greedy rule (Sec. 3.5) commits, at each slot, the candidate with the largest matching
// score sigma * cos(out, in) (Eq. pair; unit-norm in/out vectors, Sec. 3.2 and the implementation
// appendix). The fast pass computes those scores in fp32 on the matrix cores; where two of them
// are closer than the fp32 error the fp32 order can differ from the order of the scores as
// defined. For such a decision the workgroup recomputes every contender from the embedding rows
// and the fp32 weights as the definitions state them: u = e W (double, each column summed in
// row order), v = u / ||u|| rounded to fp32, cos = <o, i> / (||o|| ||i||) in double over the fp32
// vectors (each sum in index order), S = fp32(sigma * cos), z = S (+ lambda * logp with one
// fp32 rounding). Every operation is a correctly rounded IEEE double operation in a fixed order
// (products of bf16/fp32 values are exact in double; the sums of squares of double values are
// taken without fused multiply-add), so the re-scored values do not depend on how the fast pass
// tiled its work. The decision is then the lowest index among the largest re-scored z.
#pragma once

#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "common.hpp"

namespace lilicorr {

constexpr uint32_t kCertFlag = 0x80000000u;  // table entry, low word: the row was flagged
constexpr uint32_t kArgMask = 0xffu;         // table entry, low word: the fp32 argmax

// Vectors projected per sweep over a weight matrix: up to kSweepVectors per group of d threads.
constexpr int kSweepVectors = 8;

// LDS bytes of the re-scoring scratch for a workgroup of `nthreads` threads at width d.
inline size_t cert_scratch_bytes(int d, int nthreads) {
  const int nv = kSweepVectors * (nthreads / d);  // vectors per sweep
  return (size_t)nv * d * 8            // u: raw projections of one sweep
         + (size_t)(3 * nv + 2) * 8    // norms, <o, i>, <i, i>, <o, o>
         + (size_t)(nv + 1) * d * 4    // v: the out vector and the sweep's in vectors (fp32)
         + (size_t)nv * d * 2          // the sweep's embedding rows (bf16)
         + (size_t)64 * 4 * 3;         // re-scored S and z per candidate, contender list
}

__device__ __forceinline__ double bf16_to_double(uint16_t b) {
  return (double)__uint_as_float((uint32_t)b << 16);
}

// sum_j u_j^2 in index order, each square rounded before it is added
__device__ __forceinline__ double sum_squares_in_order(const double* u, int d) {
#pragma clang fp contract(off)
  double s = 0.0;
#pragma unroll 16
  for (int j = 0; j < d; ++j) s = s + u[j] * u[j];
  return s;
}

// sum_i a_i b_i in index order over fp32 values (each product exact in double)
__device__ __forceinline__ double dot_in_order(const float* a, const float* b, int d) {
  double s = 0.0;
#pragma unroll 16
  for (int i = 0; i < d; ++i) s = fma((double)a[i], (double)b[i], s);
  return s;
}

// u[v][j] = sum_i e_v[i] W[i][j] in double, i ascending (each product exact), for the vectors of
// one sweep: vector v belongs to thread group v % vp (vp = nthreads / d) at slot v / vp, and
// thread group g = tid / d takes column j = tid % d of its group's vectors, so every weight row
// is read once per sweep however many vectors share it. es holds the rows as
// [vp][d][kSweepVectors] bf16 (slots without a vector hold zeros), so one 16-byte LDS read gives
// a row element of all of a group's vectors; NV (a power of two, at least the vectors per group)
// accumulators run. The weight rows run four 8-row batches ahead of the sums, and each row's LDS
// read one row ahead (each thread's sums are sequential chains: memory latency bounds a sweep).
template <int NV>
__device__ __forceinline__ void project_sweep(double* __restrict__ u, const uint16_t* es, int nv,
                                              const float* __restrict__ W, int d, int tid,
                                              int vp) {
  typedef unsigned int u4 __attribute__((ext_vector_type(4)));
  constexpr int kRows = 8, kAhead = 4;
  const int g = tid / d, j = tid - g * d;
  if (g >= vp) return;
  const u4* eg = reinterpret_cast<const u4*>(es) + (size_t)g * d;
  double acc[NV];
#pragma unroll
  for (int v = 0; v < NV; ++v) acc[v] = 0.0;
  // row offsets go in the scalar offset of buffer loads, so a load needs no address registers
  const __amdgpu_buffer_rsrc_t rsrc = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<float*>(W), (short)0, d * d * (int)sizeof(float), 0x00020000);
  const uint32_t col = (uint32_t)j * 4u;
  float w[kAhead][kRows];
  auto load = [&](int slot, int i0) {
#pragma unroll
    for (int q = 0; q < kRows; ++q)
      w[slot][q] = __builtin_bit_cast(
          float, __builtin_amdgcn_raw_buffer_load_b32(rsrc, col, (uint32_t)((i0 + q) * d) * 4u, 0));
  };
#pragma unroll
  for (int s = 0; s < kAhead - 1; ++s)
    if (s * kRows < d) load(s, s * kRows);
  for (int i0 = 0; i0 < d; i0 += kAhead * kRows) {
#pragma unroll
    for (int s = 0; s < kAhead; ++s) {
      const int ib = i0 + s * kRows;
      if (ib < d) {
        const int ahead = ib + (kAhead - 1) * kRows;
        if (ahead < d) load((s + kAhead - 1) % kAhead, ahead);
        u4 e_next = eg[ib];
#pragma unroll
        for (int q = 0; q < kRows; ++q) {
          const u4 e = e_next;
          if (q + 1 < kRows) e_next = eg[ib + q + 1];
          const double wq = (double)w[s][q];
#pragma unroll
          for (int v = 0; v < NV; ++v) {
            const uint32_t pair = e[v / 2];
            const uint16_t b = (uint16_t)(v % 2 ? pair >> 16 : pair & 0xffffu);
            acc[v] = fma(bf16_to_double(b), wq, acc[v]);
          }
          __builtin_amdgcn_sched_barrier(0);
        }
      }
    }
  }
#pragma unroll
  for (int v = 0; v < NV; ++v) {
    const int vec = g + v * vp;
    if (vec < nv) u[vec * d + j] = acc[v];
  }
}

// project_sweep with the fewest accumulators that cover nv vectors (a choice the whole workgroup
// makes alike)
__device__ __forceinline__ void project_vectors(double* u, const uint16_t* es, int nv,
                                                const float* W, int d, int tid, int vp) {
  const int per = (nv + vp - 1) / vp;
  if (per <= 1) project_sweep<1>(u, es, nv, W, d, tid, vp);
  else if (per <= 2) project_sweep<2>(u, es, nv, W, d, tid, vp);
  else if (per <= 4) project_sweep<4>(u, es, nv, W, d, tid, vp);
  else project_sweep<8>(u, es, nv, W, d, tid, vp);
}

// Re-decides one slot among the contenders in `mask` (bit k: candidate k of the slot). Called by
// every thread of the workgroup with the same arguments; returns the decision in every thread.
//   a_out     the anchor's out vector when the slot is slot 0 with an anchor, else nullptr
//   out_id    otherwise: the embedding row of the previous slot's committed candidate
//   slot_ids  [K] candidate ids of this slot; slot_lp [K] their log-probabilities
//   arg32     the fp32 pass's decision; dlq receives z[new] - z[arg32] (re-scored values)
//   s_row     [K] pair-score output row to overwrite for the contenders, or nullptr
//   w_in, w_out  fp32 weights [d][d], row-major (row = input dimension)
__device__ __forceinline__ int certify_decision(
    const float* a_out, int32_t out_id, const int32_t* slot_ids, const float* slot_lp,
    uint64_t mask, int arg32, const uint16_t* __restrict__ E, int64_t V, int d,
    const float* __restrict__ w_in, const float* __restrict__ w_out, float sigma, float lambda,
    float* s_row, unsigned char* scratch, int tid, int nthreads, float& dlq) {
  const int vp = nthreads / d;           // column groups (>= 1: d <= nthreads)
  const int nv = kSweepVectors * vp;     // vectors per sweep
  double* u = reinterpret_cast<double*>(scratch);   // [nv][d]
  double* nrm = u + nv * d;                         // [nv]
  double* ab = nrm + nv;                            // [nv]
  double* bb = ab + nv;                             // [nv]
  double* aa = bb + nv;                             // [1] (+1 pad)
  float* vout = reinterpret_cast<float*>(aa + 2);   // [d]
  float* vc = vout + d;                             // [nv][d]
  uint16_t* es = reinterpret_cast<uint16_t*>(vc + nv * d);  // [nv][d]
  float* sr = reinterpret_cast<float*>(es + nv * d);        // [64]
  float* zr = sr + 64;                              // [64]
  int* list = reinterpret_cast<int*>(zr + 64);      // [64] contenders in increasing index

  // embedding row of sweep vector v into es, laid out for project_sweep (an id outside the table
  // is a zero row)
  auto stage_row = [&](int v, int32_t id) {
    const bool in = id >= 0 && id < V;
    uint16_t* dst = es + ((size_t)(v % vp) * d) * kSweepVectors + v / vp;
    for (int i = tid; i < d; i += nthreads)
      dst[(size_t)i * kSweepVectors] = in ? E[(int64_t)id * d + i] : 0;
  };

  const int ncont = __popcll(mask);
  if (tid < 64 && ((mask >> tid) & 1ull)) list[__popcll(mask & ((1ull << tid) - 1ull))] = tid;
  if (a_out) {
    for (int j = tid; j < d; j += nthreads) vout[j] = a_out[j];
  } else {
    // the out vector: v = u / ||u|| rounded to fp32, u = e W_out
    for (int c = 0; c < nv; ++c) stage_row(c, c == 0 ? out_id : -1);
    __syncthreads();
    project_vectors(u, es, 1, w_out, d, tid, vp);
    __syncthreads();
    if (tid == 0) nrm[0] = sqrt(sum_squares_in_order(u, d));
    __syncthreads();
    for (int j = tid; j < d; j += nthreads) vout[j] = nrm[0] > 0.0 ? (float)(u[j] / nrm[0]) : 0.f;
  }
  __syncthreads();
  if (tid == 0) *aa = dot_in_order(vout, vout, d);

  for (int base = 0; base < ncont; base += nv) {
    const int nb = ncont - base < nv ? ncont - base : nv;
    for (int c = 0; c < nv; ++c) stage_row(c, c < nb ? slot_ids[list[base + c]] : -1);
    __syncthreads();
    project_vectors(u, es, nb, w_in, d, tid, vp);
    __syncthreads();
    if (tid < nb) nrm[tid] = sqrt(sum_squares_in_order(u + tid * d, d));
    __syncthreads();
    for (int idx = tid; idx < nb * d; idx += nthreads) {
      const double nr = nrm[idx / d];
      vc[idx] = nr > 0.0 ? (float)(u[idx] / nr) : 0.f;
    }
    __syncthreads();
    if (tid < 2 * nb) {
      const int ci = tid >> 1;
      if (tid & 1) bb[ci] = dot_in_order(vc + ci * d, vc + ci * d, d);
      else ab[ci] = dot_in_order(vout, vc + ci * d, d);
    }
    __syncthreads();
    if (tid < nb) {
      const int k = list[base + tid];
      const double a2 = *aa, b2 = bb[tid];
      const double c = (a2 == 0.0 || b2 == 0.0) ? 0.0 : ab[tid] / (sqrt(a2) * sqrt(b2));
      const float sv = (float)((double)sigma * c);
      sr[k] = sv;
      zr[k] = lambda != 0.f ? fmaf(lambda, slot_lp[k], sv) : sv;
    }
    __syncthreads();
  }
  int best = list[0];
  for (int i = 1; i < ncont; ++i) {
    const int k = list[i];
    if (zr[k] > zr[best]) best = k;
  }
  dlq = best == arg32 ? 0.f : zr[best] - zr[arg32];
  if (s_row && tid < ncont) s_row[list[tid]] = sr[list[tid]];
  __syncthreads();  // the scratch is reused by the next decision
  return best;
}

}  // namespace lilicorr
