// The exact max-path decode of the decode-rule appendix: the path maximising the sum of its
// matching terms, Eq. (pathscore), g(c) = P_0[c_0] + sum_t phi(t-1, c_{t-1}, c_t), by dynamic
// programming in O(B K^2), and the local log-likelihoods of Eq. (localar) along that path.
//
// One workgroup per request. Its score matrices are staged into LDS when they fit. Wave 0 runs
// the left-to-right sweep with lane k holding the best score of a path ending at candidate k:
// at each slot it scans the K predecessors in order (a strict '>' keeps the lowest index on
// ties), in fp32 with one rounding per addition, and stores each lane's predecessor as a byte in
// LDS. One lane picks the best final candidate (lowest index on ties) and traces the
// predecessors back; then groups of 16, 32 or 64 lanes evaluate logq for all slots in parallel.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "common.hpp"
#include "lilicorr.h"

namespace lilicorr {
namespace {

constexpr int kViterbiThreads = 256;
constexpr int64_t kMaxSlots = 8192;
constexpr int64_t kMaxBackPointers = 65536;  // B * K bytes of predecessors in LDS
constexpr size_t kStageBytes = 64 * 1024;    // S[n] is staged when it fits

// v of `lane` (readlane reads the lane whatever the execution mask)
__device__ __forceinline__ float lane_value(float v, int lane) {
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), lane));
}

template <int G>
__global__ __launch_bounds__(kViterbiThreads) void viterbi_walk_kernel(
    const float* __restrict__ S, const float* __restrict__ S0, const float* __restrict__ logp,
    const int32_t* __restrict__ ids, int64_t B, int K, float lambda, bool stage,
    int32_t* __restrict__ draft, int32_t* __restrict__ choice, float* __restrict__ logq,
    float* __restrict__ score) {
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  uint8_t* from = smem;                       // [B][K] predecessors
  uint8_t* path = from + B * K;               // [B]
  float* s_lds = reinterpret_cast<float*>(smem + ((B * K + B + 15) / 16) * 16);  // [B-1][K][K]

  const int64_t n = blockIdx.x;
  const int tid = threadIdx.x;
  const int64_t per_req = (B - 1) * (int64_t)K * K;
  const float* Sn = S ? S + n * per_req : nullptr;
  const float* lpn = logp + n * B * K;
  const bool use_lp = lambda != 0.f;
  if (stage && per_req > 0) stage_words(s_lds, Sn, per_req, tid, kViterbiThreads);
  __syncthreads();
  const float* Sv = stage ? s_lds : Sn;

  if (tid < kWave) {
    const int k = tid;
    const bool live = k < K;
    float best = -__builtin_inff();
    if (live) {
      best = S0 ? S0[n * K + k] : 0.f;
      if (use_lp) best = fmaf(lambda, lpn[k], best);
    }
    for (int64_t t = 1; t < B; ++t) {
      const float* St = Sv + (t - 1) * (int64_t)K * K;
      float bv = -__builtin_inff();
      int bp = 0;
      if (live) {
        bv = lane_value(best, 0) + St[k];
        for (int p = 1; p < K; ++p) {
          const float v = lane_value(best, p) + St[p * K + k];
          if (v > bv) {
            bv = v;
            bp = p;
          }
        }
        if (use_lp) bv = fmaf(lambda, lpn[t * K + k], bv);
        from[t * K + k] = (uint8_t)bp;
      }
      best = bv;
    }
    // best final candidate (lowest index on ties), then the trace back
    int c = 0;
    float g = lane_value(best, 0);
    for (int kk = 1; kk < K; ++kk) {
      const float v = lane_value(best, kk);
      if (v > g) {
        g = v;
        c = kk;
      }
    }
    if (k == 0) {
      if (score) score[n] = g;
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
  constexpr int kGroups = kViterbiThreads / G;
  const bool live = j < K;
  for (int64_t base = 0; base < B; base += kGroups) {
    const int64_t t = base + group;
    float z = 0.f;
    int ct = 0;
    if (t < B) {
      ct = path[t];
      if (live) {
        z = t == 0 ? (S0 ? S0[n * K + j] : 0.f) : Sv[((t - 1) * K + path[t - 1]) * (int64_t)K + j];
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
      draft[n * B + t] = ids[(n * B + t) * K + ct];
      if (choice) choice[n * B + t] = ct;
      if (logq) logq[n * B + t] = (zc - m) - logf(s);
    }
  }
}

template <int G>
void launch_viterbi(int64_t N, size_t lds, hipStream_t stream, const float* S, const float* S0,
                    const float* logp, const int32_t* ids, int64_t B, int K, float lambda,
                    bool stage, int32_t* draft, int32_t* choice, float* logq, float* score) {
  static const hipError_t attr = hipFuncSetAttribute(
      reinterpret_cast<const void*>(viterbi_walk_kernel<G>),
      hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
  (void)attr;
  hipLaunchKernelGGL(viterbi_walk_kernel<G>, dim3((unsigned)N), dim3(kViterbiThreads), lds, stream,
                     S, S0, logp, ids, B, K, lambda, stage, draft, choice, logq, score);
}

}  // namespace
}  // namespace lilicorr

using namespace lilicorr;

extern "C" lilicorr_status lilicorr_viterbi_walk(const float* S, const float* S0,
                                                 const float* logp, const int32_t* ids, int64_t N,
                                                 int64_t B, int K, float logp_weight,
                                                 int32_t* draft, int32_t* choice, float* logq,
                                                 float* score, hipStream_t stream) {
  if (!logp || !ids || !draft) return LILICORR_ERR_INVALID_ARG;
  if (N < 1 || B < 1 || K < 1) return LILICORR_ERR_INVALID_ARG;
  if (B > 1 && !S) return LILICORR_ERR_INVALID_ARG;
  if (!isfinite(logp_weight)) return LILICORR_ERR_INVALID_ARG;
  if (K > 64 || B > kMaxSlots || B * K > kMaxBackPointers || N > 0x7fffffffll)
    return LILICORR_ERR_UNSUPPORTED;
  if ((S && !aligned16(S)) || (S0 && !aligned16(S0)) || !aligned16(logp) || !aligned16(ids) ||
      !aligned16(draft) || (choice && !aligned16(choice)) || (logq && !aligned16(logq)) ||
      (score && !aligned16(score)))
    return LILICORR_ERR_ALIGNMENT;
  const size_t bp_bytes = ((size_t)(B * K + B) + 15) / 16 * 16;
  const size_t s_bytes = (size_t)(B - 1) * K * K * sizeof(float);
  const bool stage = B > 1 && s_bytes <= kStageBytes;
  const size_t lds = bp_bytes + (stage ? s_bytes : 0);
  if (K <= 16)
    launch_viterbi<16>(N, lds, stream, S, S0, logp, ids, B, K, logp_weight, stage, draft, choice,
                       logq, score);
  else if (K <= 32)
    launch_viterbi<32>(N, lds, stream, S, S0, logp, ids, B, K, logp_weight, stage, draft, choice,
                       logq, score);
  else
    launch_viterbi<64>(N, lds, stream, S, S0, logp, ids, B, K, logp_weight, stage, draft, choice,
                       logq, score);
  return launch_status();
}
