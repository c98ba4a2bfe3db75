// Step 4 of the path: greedy left-to-right walk over the candidate lattice (Sec. 3.5) with the
// local log-likelihood of Eq. (localar).
//
// One workgroup per request. Everything a request's walk reads (its score matrices S[n], the
// candidate ids, the anchor scores and, when they are weighted in, the drafter log-probabilities)
// is first staged into LDS with coalesced loads, so the B dependent argmax steps touch only LDS
// and registers; lane k of wave 0 owns candidate k, and the max / sum reductions run on DPP.
// The outputs of all slots are written at the end with one coalesced store each.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "common.hpp"
#include "lilicorr.h"

namespace lilicorr {
namespace {

constexpr int kWalkThreads = 256;
constexpr size_t kWalkLdsMax = 96 * 1024;

struct WalkPlan {
  size_t s_bytes, ids_bytes, lp_bytes, out_bytes;
  int stage_s, stage_ids;
  size_t lds() const {
    return (stage_s ? s_bytes : 0) + (stage_ids ? ids_bytes + lp_bytes : 0) + out_bytes;
  }
};

inline WalkPlan walk_plan(int64_t B, int K, bool use_logp) {
  WalkPlan p;
  p.s_bytes = (size_t)(B - 1) * K * K * sizeof(float);
  p.ids_bytes = (size_t)B * K * sizeof(int32_t);
  p.lp_bytes = use_logp ? (size_t)B * K * sizeof(float) : 0;
  p.out_bytes = B <= 1024 ? (size_t)B * 2 * sizeof(int32_t) + (size_t)B * sizeof(float) : 0;
  p.stage_ids = p.ids_bytes + p.lp_bytes + p.out_bytes <= kWalkLdsMax / 2;
  p.stage_s = B > 1 && p.s_bytes + (p.stage_ids ? p.ids_bytes + p.lp_bytes : 0) + p.out_bytes <= kWalkLdsMax;
  return p;
}

__global__ __launch_bounds__(kWalkThreads) void greedy_walk_kernel(
    const float* __restrict__ S, const float* __restrict__ S0, const float* __restrict__ logp,
    const int32_t* __restrict__ ids, int64_t B, int K, float lambda, WalkPlan plan,
    int32_t* __restrict__ draft, int32_t* __restrict__ choice, float* __restrict__ logq) {
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  const int64_t n = blockIdx.x;
  const int64_t per_req = (B - 1) * (int64_t)K * K;
  const float* Sn = S ? S + n * per_req : nullptr;
  const int32_t* idn = ids + n * B * K;
  const float* lpn = logp + n * B * K;
  const bool use_lp = lambda != 0.f;

  unsigned char* p = smem;
  float* s_lds = reinterpret_cast<float*>(p);
  if (plan.stage_s) p += plan.s_bytes;
  int32_t* id_lds = reinterpret_cast<int32_t*>(p);
  float* lp_lds = reinterpret_cast<float*>(p + plan.ids_bytes);
  if (plan.stage_ids) p += plan.ids_bytes + plan.lp_bytes;
  int32_t* o_draft = reinterpret_cast<int32_t*>(p);
  int32_t* o_choice = o_draft + B;
  float* o_logq = reinterpret_cast<float*>(o_choice + B);
  const bool out_lds = plan.out_bytes > 0;

  if (plan.stage_s) stage_words(s_lds, Sn, per_req, threadIdx.x, kWalkThreads);
  if (plan.stage_ids) {
    stage_words(id_lds, idn, B * K, threadIdx.x, kWalkThreads);
    if (use_lp) stage_words(lp_lds, lpn, B * K, threadIdx.x, kWalkThreads);
  }
  __syncthreads();

  if (threadIdx.x < kWave) {
    const int lane = lane_id();
    const bool live = lane < K;
    int prev = 0;
    for (int64_t t = 0; t < B; ++t) {
      float pair = 0.f;
      if (live) {
        if (t == 0) {
          pair = S0 ? S0[n * K + lane] : 0.f;
        } else {
          const int64_t off = ((t - 1) * K + prev) * (int64_t)K + lane;
          pair = plan.stage_s ? s_lds[off] : Sn[off];
        }
      }
      float z = pair;
      if (use_lp && live)
        z = fmaf(lambda, plan.stage_ids ? lp_lds[t * K + lane] : lpn[t * K + lane], pair);
      if (!live) z = -__builtin_inff();
      const float m = wave_max_dpp(z);
      int c = __ffsll((long long)__ballot(live && z == m)) - 1;
      if (c < 0) c = 0;  // only reachable with NaN scores; keeps every access in bounds
      const float s = wave_sum_dpp(live ? expf(z - m) : 0.f);
      const int32_t tok = plan.stage_ids ? id_lds[t * K + c] : idn[t * K + c];
      if (lane == 0) {
        const float lq = -logf(s);
        if (out_lds) {
          o_draft[t] = tok;
          o_choice[t] = c;
          o_logq[t] = lq;
        } else {
          draft[n * B + t] = tok;
          if (choice) choice[n * B + t] = c;
          if (logq) logq[n * B + t] = lq;
        }
      }
      prev = c;
    }
  }
  if (out_lds) {
    __syncthreads();
    for (int64_t t = threadIdx.x; t < B; t += kWalkThreads) {
      draft[n * B + t] = o_draft[t];
      if (choice) choice[n * B + t] = o_choice[t];
      if (logq) logq[n * B + t] = o_logq[t];
    }
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
  const WalkPlan plan = walk_plan(B, K, logp_weight != 0.f);
  static const hipError_t attr = hipFuncSetAttribute(
      reinterpret_cast<const void*>(greedy_walk_kernel),
      hipFuncAttributeMaxDynamicSharedMemorySize, (int)kWalkLdsMax);
  (void)attr;
  hipLaunchKernelGGL(greedy_walk_kernel, dim3((unsigned)N), dim3(kWalkThreads), plan.lds(), stream,
                     S, S0, logp, ids, B, K, logp_weight, plan, draft, choice, logq);
  return launch_status();
}
