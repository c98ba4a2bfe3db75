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

// LDS bytes of the re-scoring scratch for a workgroup of `nthreads` threads at width d.
inline size_t cert_scratch_bytes(int d, int nthreads) {
  const int vp = nthreads / d;
  return (size_t)vp * d * 8            // u: raw projections of one pass
         + (size_t)(3 * vp + 2) * 8    // norms, <o, i>, <i, i>, <o, o>
         + (size_t)(vp + 1) * d * 4    // v: the out vector and the pass's in vectors (fp32)
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
  const int vp = nthreads / d;  // vectors projected per pass (>= 2 for d <= 256)
  double* u = reinterpret_cast<double*>(scratch);  // [vp][d]
  double* nrm = u + vp * d;                         // [vp]
  double* ab = nrm + vp;                            // [vp]
  double* bb = ab + vp;                             // [vp]
  double* aa = bb + vp;                             // [1] (+1 pad)
  float* vout = reinterpret_cast<float*>(aa + 2);   // [d]
  float* vc = vout + d;                             // [vp][d]
  float* sr = vc + vp * d;                          // [64]
  float* zr = sr + 64;                              // [64]
  int* list = reinterpret_cast<int*>(zr + 64);      // [64] contenders in increasing index

  const int ncont = __popcll(mask);
  const bool anchored = a_out != nullptr;
  if (tid < 64 && ((mask >> tid) & 1ull)) list[__popcll(mask & ((1ull << tid) - 1ull))] = tid;
  if (anchored)
    for (int j = tid; j < d; j += nthreads) vout[j] = a_out[j];
  __syncthreads();

  const int first = anchored ? 0 : 1;  // item 0 is the out vector unless the anchor gives it
  const int total = first + ncont;
  const int vi = tid / d, j = tid % d;
  for (int base = 0; base < total; base += vp) {
    const int nvp = total - base < vp ? total - base : vp;
    const int item = base + vi;
    const bool is_out = !anchored && item == 0;
    if (vi < nvp) {
      const int32_t id = is_out ? out_id : slot_ids[list[item - first]];
      const float* W = is_out ? w_out : w_in;
      double acc = 0.0;
      if (id >= 0 && id < V) {  // an id outside the table is a zero row
        const uint16_t* e = E + (int64_t)id * d;
#pragma unroll 8
        for (int i = 0; i < d; ++i) acc = fma(bf16_to_double(e[i]), (double)W[(int64_t)i * d + j], acc);
      }
      u[vi * d + j] = acc;
    }
    __syncthreads();
    if (tid < nvp) nrm[tid] = sqrt(sum_squares_in_order(u + tid * d, d));
    __syncthreads();
    if (vi < nvp) {
      const double nr = nrm[vi];
      const float v = nr > 0.0 ? (float)(u[vi * d + j] / nr) : 0.f;
      if (is_out) vout[j] = v;
      else vc[vi * d + j] = v;
    }
    __syncthreads();
    if (base == 0 && tid == 2 * vp) *aa = dot_in_order(vout, vout, d);
    if (tid < 2 * nvp && base + (tid >> 1) >= first) {
      const int ci = tid >> 1;
      if (tid & 1) bb[ci] = dot_in_order(vc + ci * d, vc + ci * d, d);
      else ab[ci] = dot_in_order(vout, vc + ci * d, d);
    }
    __syncthreads();
    if (tid < nvp && base + tid >= first) {
      const int k = list[base + tid - first];
      const double a2 = *aa, b2 = bb[tid];
      const double c = (a2 == 0.0 || b2 == 0.0) ? 0.0 : ab[tid] / (sqrt(a2) * sqrt(b2));
      const float s = (float)((double)sigma * c);
      sr[k] = s;
      zr[k] = lambda != 0.f ? fmaf(lambda, slot_lp[k], s) : s;
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
