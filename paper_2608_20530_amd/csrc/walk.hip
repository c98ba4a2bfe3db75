// Step 4 of the path: greedy left-to-right walk over the candidate lattice (Sec. 3.5) with the
// local log-likelihood of Eq. (localar).
//
// The walk's choice at slot t depends only on its choice at t-1, through one row of S. So every
// row the walk could visit, (slot t, previous choice p), is resolved first, all in parallel: its
// argmax (lowest index on ties) and its local log-likelihood -log sum_k exp(z_k - max z). Each row
// is handled by a group of 16, 32 or 64 lanes (one lane per candidate) with DPP butterflies, and
// the results go to an LDS table. One lane then follows the table, one LDS read per slot, and the
// whole workgroup writes the slots' outputs. One workgroup per request; slots are processed in
// segments whose table fits in LDS. Workgroups have 256 threads at K <= 16 (one round of row loads
// covers a 16-slot block's 241 rows) and 512 above (at K = 32 the 481 rows take two rounds of
// loads instead of four; 1024 threads would cap the registers below what 16 rows in flight per
// lane need).
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "common.hpp"
#include "lilicorr.h"

namespace lilicorr {
namespace {

// threads per workgroup for groups of G lanes
template <int G>
__host__ __device__ constexpr int walk_threads() { return G <= 16 ? 256 : 512; }
constexpr int kSegRows = 2048;  // table rows per segment (slots per segment: kSegRows / K)
constexpr int kRowBatch = 16;   // rows per group whose loads are issued together

template <int G>
__global__ __launch_bounds__(walk_threads<G>()) void greedy_walk_kernel(
    const float* __restrict__ S, const float* __restrict__ S0, const float* __restrict__ logp,
    const int32_t* __restrict__ ids, int64_t B, int K, float lambda,
    int32_t* __restrict__ draft, int32_t* __restrict__ choice, float* __restrict__ logq) {
  // row table: low 32 bits the argmax, high 32 bits the fp32 local log-likelihood
  __shared__ uint64_t table[kSegRows + 1];
  __shared__ int32_t seg_choice[kSegRows];
  __shared__ float seg_logq[kSegRows];

  constexpr int kWalkThreads = walk_threads<G>();
  const int64_t n = blockIdx.x;
  const int tid = threadIdx.x;
  const int j = tid % G;                 // candidate index within the row
  const int group = tid / G;
  constexpr int kGroups = kWalkThreads / G;
  const bool live = j < K;
  const bool use_lp = lambda != 0.f;
  const float* Sn = S ? S + n * (B - 1) * (int64_t)K * K : nullptr;
  const float* lpn = logp + n * B * K;
  const int64_t T = kSegRows / K > 0 ? kSegRows / K : 1;  // slots per segment

  int c = 0;  // the walk's current choice (used by thread 0)
  for (int64_t t0 = 0; t0 < B; t0 += T) {
    const int64_t t1 = t0 + T < B ? t0 + T : B;
    // global rows: 0 is slot 0; 1 + (t-1) K + p is slot t >= 1 after choice p
    const int64_t rb = t0 == 0 ? 0 : 1 + (t0 - 1) * K;
    const int64_t re = 1 + (t1 - 1) * K;
    // the trip count is the same for every thread, so whole waves stay converged for the
    // butterflies and ballots
    for (int64_t base = rb; base < re; base += (int64_t)kRowBatch * kGroups) {
      float z[kRowBatch];
#pragma unroll
      for (int u = 0; u < kRowBatch; ++u) {
        const int64_t row = base + group + (int64_t)u * kGroups;
        float v = -__builtin_inff();
        if (live && row < re) {
          if (row == 0) {
            v = S0 ? S0[n * K + j] : 0.f;
            if (use_lp) v = fmaf(lambda, lpn[j], v);
          } else {
            v = Sn[(row - 1) * K + j];
            if (use_lp) v = fmaf(lambda, lpn[(1 + (row - 1) / K) * K + j], v);
          }
        }
        z[u] = v;
      }
#pragma unroll
      for (int u = 0; u < kRowBatch; ++u) {
        const int64_t row = base + group + (int64_t)u * kGroups;
        int arg;
        float lq;
        resolve_row<G>(z[u], live, arg, lq);
        if (j == 0 && row < re) table[row - rb] = table_entry(arg, lq);
      }
    }
    __syncthreads();
    if (tid == 0) {
      for (int64_t t = t0; t < t1; ++t) {
        const int64_t row = t == 0 ? 0 : 1 + (t - 1) * K + c;
        const uint64_t e = table[row - rb];
        c = (int)(uint32_t)e;
        seg_choice[t - t0] = c;
        seg_logq[t - t0] = __uint_as_float((uint32_t)(e >> 32));
      }
    }
    __syncthreads();
    for (int64_t t = t0 + tid; t < t1; t += kWalkThreads) {
      const int ct = seg_choice[t - t0];
      draft[n * B + t] = ids[(n * B + t) * K + ct];
      if (choice) choice[n * B + t] = ct;
      if (logq) logq[n * B + t] = seg_logq[t - t0];
    }
    __syncthreads();
  }
}

}  // namespace
}  // namespace lilicorr

using namespace lilicorr;

extern "C" lilicorr_status lilicorr_greedy_walk(const float* S, const float* S0, const float* logp,
                                                const int32_t* ids, int64_t N, int64_t B, int K,
                                                float logp_weight, int32_t* draft, int32_t* choice,
                                                float* logq, hipStream_t stream) {
  if (!logp || !ids || !draft) return LILICORR_ERR_INVALID_ARG;
  if (N < 1 || B < 1 || K < 1) return LILICORR_ERR_INVALID_ARG;
  if (B > 1 && !S) return LILICORR_ERR_INVALID_ARG;
  if (K > 64) return LILICORR_ERR_UNSUPPORTED;
  if (N > 0x7fffffffll || B > ((int64_t)1 << 40) / K) return LILICORR_ERR_UNSUPPORTED;
  if (!isfinite(logp_weight)) return LILICORR_ERR_INVALID_ARG;
  if ((S && !aligned16(S)) || (S0 && !aligned16(S0)) || !aligned16(logp) || !aligned16(ids) ||
      !aligned16(draft) || (choice && !aligned16(choice)) || (logq && !aligned16(logq)))
    return LILICORR_ERR_ALIGNMENT;
  const dim3 grid((unsigned)N);
  if (K <= 16)
    hipLaunchKernelGGL(greedy_walk_kernel<16>, grid, dim3(walk_threads<16>()), 0, stream, S, S0,
                       logp, ids, B, K, logp_weight, draft, choice, logq);
  else if (K <= 32)
    hipLaunchKernelGGL(greedy_walk_kernel<32>, grid, dim3(walk_threads<32>()), 0, stream, S, S0,
                       logp, ids, B, K, logp_weight, draft, choice, logq);
  else
    hipLaunchKernelGGL(greedy_walk_kernel<64>, grid, dim3(walk_threads<64>()), 0, stream, S, S0,
                       logp, ids, B, K, logp_weight, draft, choice, logq);
  return launch_status();
}
