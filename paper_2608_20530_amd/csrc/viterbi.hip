// The exact max-path decode of the decode-rule appendix: the path maximising the sum of its
// matching terms, Eq. (pathscore), by dynamic programming in O(B K^2), and the local
// log-likelihoods of Eq. (localar) along that path. One workgroup per request; its score
// matrices are staged into LDS when they fit (up to the 160 KB of a compute unit), and the sweep
// itself is viterbi_block.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "common.hpp"
#include "lilicorr.h"
#include "viterbi.hpp"

namespace lilicorr {
namespace {

constexpr int kViterbiThreads = 256;
constexpr int64_t kMaxSlots = 8192;
constexpr int64_t kMaxBackPointers = 65536;  // B * K bytes of predecessors in LDS
constexpr size_t kMaxLds = 160 * 1024;       // S[n] is staged (transposed) when it fits

template <int G>
__global__ __launch_bounds__(kViterbiThreads) void viterbi_walk_kernel(
    const float* __restrict__ S, const float* __restrict__ S0, const float* __restrict__ logp,
    const int32_t* __restrict__ ids, int64_t B, int K, float lambda, bool stage,
    int32_t* __restrict__ draft, int32_t* __restrict__ choice, float* __restrict__ logq,
    float* __restrict__ score) {
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  uint8_t* from = smem;                       // [B][K] predecessors
  uint8_t* path = from + B * K;               // [B]
  double* line = reinterpret_cast<double*>(smem + ((B * K + B + 15) / 16) * 16);  // [64]
  float* T = reinterpret_cast<float*>(line + kWave);  // [B-1][K][G+4] transposed scores (staged)

  const int64_t n = blockIdx.x;
  const int tid = threadIdx.x;
  const float* Sn = S ? S + n * (B - 1) * (int64_t)K * K : nullptr;
  const float* S0n = S0 ? S0 + n * K : nullptr;
  int32_t* choice_n = choice ? choice + n * B : nullptr;
  float* logq_n = logq ? logq + n * B : nullptr;
  float* score_n = score ? score + n : nullptr;
  if (stage) {
    if (B > 1) stage_transposed<G>(T, Sn, B, K, tid, kViterbiThreads);
    __syncthreads();
    viterbi_block<G, true>(T, S0n, logp + n * B * K, ids + n * B * K, B, K, lambda, from, path,
                           line, draft + n * B, choice_n, logq_n, score_n, tid, kViterbiThreads);
  } else {
    viterbi_block<G, false>(Sn, S0n, logp + n * B * K, ids + n * B * K, B, K, lambda, from,
                            path, line, draft + n * B, choice_n, logq_n, score_n, tid,
                            kViterbiThreads);
  }
}

template <int G>
void launch_viterbi(int64_t N, int64_t B, int K, hipStream_t stream, const float* S,
                    const float* S0, const float* logp, const int32_t* ids, float lambda,
                    int32_t* draft, int32_t* choice, float* logq, float* score) {
  const size_t head = ((size_t)(B * K + B) + 15) / 16 * 16 + kWave * sizeof(double);
  const size_t t_bytes = (size_t)(B - 1) * K * viterbi_stride<G>() * sizeof(float);
  const bool stage = B > 1 && head + t_bytes <= kMaxLds;
  static const hipError_t attr = hipFuncSetAttribute(
      reinterpret_cast<const void*>(viterbi_walk_kernel<G>),
      hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
  (void)attr;
  hipLaunchKernelGGL(viterbi_walk_kernel<G>, dim3((unsigned)N), dim3(kViterbiThreads),
                     head + (stage ? t_bytes : 0), stream, S, S0, logp, ids, B, K, lambda, stage,
                     draft, choice, logq, score);
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
  if (K <= 16)
    launch_viterbi<16>(N, B, K, stream, S, S0, logp, ids, logp_weight, draft, choice, logq, score);
  else if (K <= 32)
    launch_viterbi<32>(N, B, K, stream, S, S0, logp, ids, logp_weight, draft, choice, logq, score);
  else
    launch_viterbi<64>(N, B, K, stream, S, S0, logp, ids, logp_weight, draft, choice, logq, score);
  return launch_status();
}
