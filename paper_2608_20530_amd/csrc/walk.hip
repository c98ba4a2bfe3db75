// Step 4 of the path: greedy left-to-right walk over the candidate lattice (Sec. 3.5) with the
// local log-likelihood of Eq. (localar).
//
// One workgroup per request. The request's score matrices S[n] ((B-1) x K x K fp32) are staged
// into LDS with coalesced loads when they fit, so the B-1 dependent argmax steps read LDS instead
// of making a round trip to HBM each. Lane k of wave 0 owns candidate k; the argmax is a wave max
// followed by a ballot for the lowest attaining lane.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "common.hpp"
#include "lilicorr.h"

namespace lilicorr {
namespace {

constexpr int kWalkThreads = 256;
constexpr size_t kWalkLdsMax = 64 * 1024;

__global__ __launch_bounds__(kWalkThreads) void greedy_walk_kernel(
    const float* __restrict__ S, const float* __restrict__ S0, const float* __restrict__ logp,
    const int32_t* __restrict__ ids, int64_t B, int K, float lambda, int staged,
    int32_t* __restrict__ draft, int32_t* __restrict__ choice, float* __restrict__ logq) {
  extern __shared__ float lds[];
  const int64_t n = blockIdx.x;
  const int64_t per_req = (B - 1) * (int64_t)K * K;
  const float* Sn = S ? S + n * per_req : nullptr;
  if (staged) {
    for (int64_t i = threadIdx.x; i < per_req; i += kWalkThreads) lds[i] = Sn[i];
    __syncthreads();
  }
  if (threadIdx.x >= kWave) return;
  const int lane = lane_id();
  const bool live = lane < K;
  int prev = 0;
  for (int64_t t = 0; t < B; ++t) {
    float pair = 0.f;
    if (live) {
      if (t == 0) {
        pair = S0 ? S0[n * K + lane] : 0.f;
      } else {
        int64_t off = ((t - 1) * K + prev) * (int64_t)K + lane;
        pair = staged ? lds[off] : Sn[off];
      }
    }
    float z = pair;
    if (lambda != 0.f) z = fmaf(lambda, live ? logp[(n * B + t) * K + lane] : 0.f, pair);
    if (!live) z = -__builtin_inff();
    float m = wave_max(z);
    int c = __ffsll((long long)__ballot(live && z == m)) - 1;
    if (c < 0) c = 0;  // only reachable with NaN scores; keeps every access in bounds
    float e = live ? expf(z - m) : 0.f;
    float s = wave_sum(e);
    if (lane == 0) {
      draft[n * B + t] = ids[(n * B + t) * K + c];
      if (choice) choice[n * B + t] = c;
      if (logq) logq[n * B + t] = -logf(s);
    }
    prev = c;
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
  const size_t bytes = (size_t)(B - 1) * K * K * sizeof(float);
  const int staged = (B > 1 && bytes <= kWalkLdsMax) ? 1 : 0;
  hipLaunchKernelGGL(greedy_walk_kernel, dim3((unsigned)N), dim3(kWalkThreads),
                     staged ? bytes : 0, stream, S, S0, logp, ids, B, K, logp_weight, staged,
                     draft, choice, logq);
  return launch_status();
}
