// Step 3 of the path: batched pair matching scores, Eq. (pair):
//   S[n][t][k][k'] = sigma * cos(out[n][t][k], in[n][t+1][k'])
// one K x K matrix per adjacent slot pair, batched over the block (Sec. 3.5), and the anchor pair
// S0[n][k'] = sigma * cos(anchor_out[n], in[n][0][k']).
//
// One wavefront per (request, pair) matrix, on the fp32 matrix cores (v_mfma_f32_16x16x4_f32):
// S is a [K x d] x [d x K] product, cut into 16 x 16 output tiles. A dot product may visit the
// vector dimension in any order, so each lane reads whole 16-byte pieces of one row: lane (r, q)
// (r = lane % 16, q = lane / 16) holds columns 4(q + 4s) .. 4(q + 4s) + 3 of left and right row r
// for s = 0, 1, ... within each chunk of 16*S4 columns, and MFMA step (s, e) contracts column
// 4(q + 4s) + e of both sides. A load instruction then covers 64 contiguous bytes of each of 16
// rows. Loads go through buffer descriptors bounded to the matrix's rows, so rows past K and
// columns past d read as zeros without touching memory; chunks alternate between two register
// sets, the next one loading while the current one is contracted. Squared norms accumulate
// alongside, per lane, and are summed over the four lanes that share a row at the end.
//
// Steps 3-4 in one pass (lilicorr_pair_walk and its certified and exact-decode forms): the same
// matrices, eight per workgroup of eight waves, then, instead of S going to memory and a walk
// kernel reading it back, each wave resolves its matrix's rows of the walk's transition table
// (or, for the exact decode, hands its scores over) and the request's last workgroup decodes
// (handover.hpp). This is the form of the one-pass decode for vectors of any width: the fused
// projection pass holds both sides' vectors in LDS, which bounds it to d <= 256.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "common.hpp"
#include "handover.hpp"
#include "lilicorr.h"
#include "projection.hpp"

namespace lilicorr {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr uint32_t kOutOfRange = 0x80000000u;  // byte offset past every descriptor's range

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rows_rsrc(const float* base, int rows, int d) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(base), (short)0,
                                           rows * d * (int)sizeof(float), 0x00020000);
}

// NB 16-row blocks of one side, S4 16-byte pieces per lane and block, for the chunk at column c0
template <int NB, int S4>
__device__ __forceinline__ void load_chunk(f32x4 (&v)[NB][S4], __amdgpu_buffer_rsrc_t rsrc,
                                           int rows, int d, int c0, int r, int q) {
#pragma unroll
  for (int bl = 0; bl < NB; ++bl)
#pragma unroll
    for (int s = 0; s < S4; ++s) {
      const int row = bl * 16 + r, col = c0 + 4 * (q + 4 * s);
      const uint32_t off =
          (row < rows && col < d) ? (uint32_t)((row * d + col) * (int)sizeof(float)) : kOutOfRange;
      v[bl][s] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(rsrc, off, 0, 0));
    }
}

template <int NBL, int NBR, int S4>
__device__ __forceinline__ void contract_chunk(f32x4 (&acc)[NBL][NBR], float (&nl)[NBL],
                                               float (&nr)[NBR], const f32x4 (&a)[NBL][S4],
                                               const f32x4 (&b)[NBR][S4]) {
#pragma unroll
  for (int s = 0; s < S4; ++s)
#pragma unroll
    for (int e = 0; e < 4; ++e)
#pragma unroll
      for (int bl = 0; bl < NBL; ++bl)
#pragma unroll
        for (int br = 0; br < NBR; ++br)
          acc[bl][br] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[bl][s][e], b[br][s][e], acc[bl][br],
                                                             0, 0, 0);
#pragma unroll
  for (int bl = 0; bl < NBL; ++bl)
#pragma unroll
    for (int s = 0; s < S4; ++s)
#pragma unroll
      for (int e = 0; e < 4; ++e) nl[bl] = fmaf(a[bl][s][e], a[bl][s][e], nl[bl]);
#pragma unroll
  for (int br = 0; br < NBR; ++br)
#pragma unroll
    for (int s = 0; s < S4; ++s)
#pragma unroll
      for (int e = 0; e < 4; ++e) nr[br] = fmaf(b[br][s][e], b[br][s][e], nr[br]);
}

// The raw dot products and squared norms of one K x K (or 1 x K) matrix, by one wave: acc[bl][br]
// is tile (bl, br) of left . right^T (lane l holds rows 4(l/16) + i, column l % 16, i = 0..3),
// nl[bl] / nr[br] the squared norm of left / right row 16 bl + l % 16 (br: 16 br + l % 16).
template <int NBL, int NBR, int S4>
__device__ __forceinline__ void matrix_dots(f32x4 (&acc)[NBL][NBR], float (&nl)[NBL],
                                            float (&nr)[NBR], const float* left, int KL,
                                            const float* right, int K, int d, int r, int q) {
  constexpr int kCols = 16 * S4;  // columns per chunk
  const __amdgpu_buffer_rsrc_t rl = rows_rsrc(left, KL, d), rr = rows_rsrc(right, K, d);
#pragma unroll
  for (int bl = 0; bl < NBL; ++bl)
#pragma unroll
    for (int br = 0; br < NBR; ++br) acc[bl][br] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int bl = 0; bl < NBL; ++bl) nl[bl] = 0.f;
#pragma unroll
  for (int br = 0; br < NBR; ++br) nr[br] = 0.f;

  // two chunks per trip through two register sets; a chunk past d loads zeros without traffic
  f32x4 a0[NBL][S4], b0[NBR][S4], a1[NBL][S4], b1[NBR][S4];
  load_chunk<NBL, S4>(a0, rl, KL, d, 0, r, q);
  load_chunk<NBR, S4>(b0, rr, K, d, 0, r, q);
  for (int c0 = 0; c0 < d; c0 += 2 * kCols) {
    load_chunk<NBL, S4>(a1, rl, KL, d, c0 + kCols, r, q);
    load_chunk<NBR, S4>(b1, rr, K, d, c0 + kCols, r, q);
    contract_chunk<NBL, NBR, S4>(acc, nl, nr, a0, b0);
    load_chunk<NBL, S4>(a0, rl, KL, d, c0 + 2 * kCols, r, q);
    load_chunk<NBR, S4>(b0, rr, K, d, c0 + 2 * kCols, r, q);
    contract_chunk<NBL, NBR, S4>(acc, nl, nr, a1, b1);
  }

  // lanes r, r+16, r+32, r+48 share row r: sum their partial norms
#pragma unroll
  for (int bl = 0; bl < NBL; ++bl) {
    nl[bl] += __shfl_xor(nl[bl], 16, kWave);
    nl[bl] += __shfl_xor(nl[bl], 32, kWave);
  }
#pragma unroll
  for (int br = 0; br < NBR; ++br) {
    nr[br] += __shfl_xor(nr[br], 16, kWave);
    nr[br] += __shfl_xor(nr[br], 32, kWave);
  }
}

// f(k, kk, S[k][kk]) for every entry of the matrix this lane holds, S = sigma * cos (a zero row
// scores 0)
template <int NBL, int NBR, typename F>
__device__ __forceinline__ void for_each_score(const f32x4 (&acc)[NBL][NBR], const float (&nl)[NBL],
                                               const float (&nr)[NBR], int KL, int K, float sigma,
                                               int r, int q, F f) {
#pragma unroll
  for (int bl = 0; bl < NBL; ++bl)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float nrow = __shfl(nl[bl], 4 * q + i, kWave);
      const int k = bl * 16 + 4 * q + i;
#pragma unroll
      for (int br = 0; br < NBR; ++br) {
        const int kk = br * 16 + r;
        if (k < KL && kk < K) {
          const float den = sqrtf(nrow) * sqrtf(nr[br]);
          f(k, kk, den > 0.f ? sigma * (acc[bl][br][i] / den) : 0.f);
        }
      }
    }
}

template <int NBL, int NBR, int S4>
__global__ __launch_bounds__(kWave) void pair_scores_kernel(
    const float* __restrict__ in_vec, const float* __restrict__ out_vec,
    const float* __restrict__ anchor_out, int64_t B, int K, int d, float sigma,
    float* __restrict__ S, float* __restrict__ S0) {
  const int lane = lane_id();
  const int r = lane & 15, q = lane >> 4;
  const int64_t n = blockIdx.y;
  const int pair = blockIdx.x;  // 0..B-2 slot pairs; B-1 is the anchor pair when given
  const bool anchor = pair == (int)(B - 1);
  const int KL = anchor ? 1 : K;
  const float* left = anchor ? anchor_out + n * d : out_vec + ((n * B + pair) * K) * (int64_t)d;
  const float* right = in_vec + ((n * B + (anchor ? 0 : pair + 1)) * K) * (int64_t)d;
  f32x4 acc[NBL][NBR];
  float nl[NBL], nr[NBR];
  matrix_dots<NBL, NBR, S4>(acc, nl, nr, left, KL, right, K, d, r, q);
  float* dst = anchor ? S0 + n * K : S + ((n * (B - 1) + pair) * K) * (int64_t)K;
  const int rstride = anchor ? 0 : K;
  for_each_score<NBL, NBR>(acc, nl, nr, KL, K, sigma, r, q,
                           [&](int k, int kk, float v) { dst[k * rstride + kk] = v; });
}

template <int NB, int S4>
void launch_pairs(dim3 grid, hipStream_t stream, const float* in_vec, const float* out_vec,
                  const float* anchor_out, int64_t B, int K, int d, float sigma, float* S,
                  float* S0) {
  hipLaunchKernelGGL((pair_scores_kernel<NB, NB, S4>), grid, dim3(kWave), 0, stream, in_vec,
                     out_vec, anchor_out, B, K, d, sigma, S, S0);
}


constexpr int kPairWaves = 8;  // matrices (waves) per workgroup of the one-pass decode

// The one-pass decode over precomputed vectors. Workgroup (x, n) holds matrices 8x .. 8x+7 of
// request n, one per wave: slot pairs 0 .. B-2, then the anchor pair when given. Waves without a
// matrix (the request's last workgroup may have fewer than eight) only take part in the
// workgroup's barriers.
template <int NB, int S4, int G, bool EXACT, bool CERT>
__global__ __launch_bounds__(kPairWaves * kWave)
__attribute__((amdgpu_waves_per_eu(NB <= 2 ? 4 : 2))) void pair_walk_kernel(
    const float* __restrict__ in_vec, const float* __restrict__ out_vec,
    const float* __restrict__ anchor_out, const float* __restrict__ logp,
    const int32_t* __restrict__ ids, const uint16_t* __restrict__ E, int64_t V, int64_t B, int K,
    int d, float sigma, float lambda, float margin, const float* __restrict__ w32, TailPlan tail,
    size_t flag_off, float* __restrict__ S, float* __restrict__ S0, int32_t* __restrict__ draft,
    int32_t* __restrict__ choice, float* __restrict__ logq, float* __restrict__ score,
    int32_t* __restrict__ rescored, uint32_t* __restrict__ counters, void* __restrict__ exchange,
    uint64_t* __restrict__ cmask) {
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  const int tid = threadIdx.x;
  const int wave = tid / kWave, lane = lane_id();
  const int r = lane & 15, q = lane >> 4;
  const int64_t n = blockIdx.y;
  const int nmat = (int)(B - 1) + (anchor_out ? 1 : 0);
  const int pair = blockIdx.x * kPairWaves + wave;
  const bool has = pair < nmat;
  const bool anchor = has && pair == (int)(B - 1);
  const int KL = anchor ? 1 : K;
  float* sw = reinterpret_cast<float*>(smem) + wave * K * K;  // [K][K] this wave's scores
  int* flag = reinterpret_cast<int*>(smem + flag_off);

  if (has) {
    const float* left = anchor ? anchor_out + n * d : out_vec + ((n * B + pair) * K) * (int64_t)d;
    const float* right = in_vec + ((n * B + (anchor ? 0 : pair + 1)) * K) * (int64_t)d;
    f32x4 acc[NB][NB];
    float nl[NB], nr[NB];
    matrix_dots<NB, NB, S4>(acc, nl, nr, left, KL, right, K, d, r, q);
    float* dst = anchor ? S0 + n * K : S + ((n * (B - 1) + pair) * K) * (int64_t)K;
    const bool keep = anchor ? S0 != nullptr : S != nullptr;
    const int rstride = anchor ? 0 : K;
    float* xn = static_cast<float*>(exchange) + n * tail.rows + (int64_t)pair * K * K;
    for_each_score<NB, NB>(acc, nl, nr, KL, K, sigma, r, q, [&](int k, int kk, float v) {
      if (keep) dst[k * rstride + kk] = v;
      if (EXACT)
        exchange_store(&xn[k * K + kk], v);  // the anchor row follows the B-1 pair blocks
      else
        sw[k * K + kk] = v;
    });
  }
  if (!EXACT) {
    __syncthreads();
    // this wave's rows: (slot pair+1, previous choice k) for its slot pair, row 0 (slot 0) for
    // the anchor pair, and row 0 in wave 0 of workgroup 0 when there is no anchor
    const bool use_lp = lambda != 0.f;
    const float* lpn = logp + n * B * K;
    const int prow = has && !anchor ? K : 0;
    const bool row0 = anchor || (anchor_out == nullptr && blockIdx.x == 0 && wave == 0);
    const int nrows = prow + (row0 ? 1 : 0);
    const int j = lane % G;
    const bool live = j < K;
    uint64_t* table_n = static_cast<uint64_t*>(exchange) + n * tail.rows;
    uint64_t* cmask_n = CERT ? cmask + n * tail.rows : nullptr;
    for (int base = 0; base < nrows; base += kWave / G) {  // the same trip count in every lane
      const int lr = base + lane / G;
      float z = 0.f;
      if (lr < nrows && live) {
        if (lr < prow) {
          z = sw[lr * K + j];
          if (use_lp) z = fmaf(lambda, lpn[(pair + 1) * K + j], z);
        } else {
          z = anchor ? sw[j] : 0.f;
          if (use_lp) z = fmaf(lambda, lpn[j], z);
        }
      }
      const int64_t grow = lr >= nrows ? -1 : (lr < prow ? 1 + (int64_t)pair * K + lr : 0);
      hand_over_row<G, CERT>(z, live, grow, lr < prow || anchor, margin, table_n, cmask_n, j);
    }
  }
  if (!take_ticket(&counters[n], gridDim.x, flag, tid, CERT && (S || S0))) return;
  TailArgs ta{n, B, V, K, d, sigma, lambda, E, w32, anchor_out, ids, logp, S, S0, draft,
              choice, logq, score, rescored, &counters[n], exchange, cmask, tail};
  finish_request<G, EXACT, CERT>(ta, smem, tid, kPairWaves * kWave);
}

// the kernel arguments after grid, LDS bytes and stream
#define PAIR_WALK_PARAMS                                                                          \
  const float *in_vec, const float *out_vec, const float *anchor_out, const float *logp,         \
      const int32_t *ids, const uint16_t *E, int64_t V, int64_t B, int K, int d, float sigma,    \
      float lambda, float margin, const float *w32, TailPlan tail, size_t flag_off, float *S,    \
      float *S0, int32_t *draft, int32_t *choice, float *logq, float *score, int32_t *rescored, \
      uint32_t *counters, void *exchange, uint64_t *cmask

// one instance per kernel, so the LDS limit is raised once for each kernel
template <int NB, int S4, int G, bool EXACT, bool CERT>
void launch_pair_walk(dim3 grid, size_t lds, hipStream_t stream, PAIR_WALK_PARAMS) {
  static const hipError_t attr = hipFuncSetAttribute(
      reinterpret_cast<const void*>(pair_walk_kernel<NB, S4, G, EXACT, CERT>),
      hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
  (void)attr;
  hipLaunchKernelGGL((pair_walk_kernel<NB, S4, G, EXACT, CERT>), grid, dim3(kPairWaves * kWave),
                     lds, stream, in_vec, out_vec, anchor_out, logp, ids, E, V, B, K, d, sigma,
                     lambda, margin, w32, tail, flag_off, S, S0, draft, choice, logq, score,
                     rescored, counters, exchange, cmask);
}
#undef PAIR_WALK_PARAMS

// validation and launch of the one-pass decode over precomputed vectors
template <bool EXACT, bool CERT>
lilicorr_status pairs_and_decode(const float* in_vec, const float* out_vec,
                                 const float* anchor_out, const float* logp, const int32_t* ids,
                                 const void* E, lilicorr_dtype e_dtype, int64_t V,
                                 const void* packed_w, int64_t N, int64_t B, int K, int d,
                                 float sigma, float logp_weight, float margin, float* S, float* S0,
                                 int32_t* draft, int32_t* choice, float* logq, float* score,
                                 int32_t* rescored, void* workspace, size_t workspace_bytes,
                                 hipStream_t stream) {
  if (!in_vec || !out_vec || !logp || !ids || !draft || !workspace) return LILICORR_ERR_INVALID_ARG;
  if (CERT && (!E || !packed_w || V < 1)) return LILICORR_ERR_INVALID_ARG;
  if (CERT && e_dtype != LILICORR_F32 && e_dtype != LILICORR_BF16) return LILICORR_ERR_INVALID_ARG;
  if (N < 1 || B < 1 || K < 1 || d < 1) return LILICORR_ERR_INVALID_ARG;
  if (!isfinite(sigma) || !isfinite(logp_weight)) return LILICORR_ERR_INVALID_ARG;
  if (CERT && !(isfinite(margin) && margin >= 0.f)) return LILICORR_ERR_INVALID_ARG;
  // the re-scoring reads bf16 rows and projects one vector per d threads of the workgroup
  if (CERT && (e_dtype != LILICORR_BF16 || d > kPairWaves * kWave)) return LILICORR_ERR_UNSUPPORTED;
  if (d % 16 != 0 || d > 1024 || !decode_shape_ok(N, B, K, EXACT)) return LILICORR_ERR_UNSUPPORTED;
  if (N > 65535) return LILICORR_ERR_UNSUPPORTED;
  if (!aligned16(in_vec) || !aligned16(out_vec) || !aligned16(logp) || !aligned16(ids) ||
      !aligned16(draft) || !aligned16(workspace) || (anchor_out && !aligned16(anchor_out)) ||
      (S && !aligned16(S)) || (S0 && !aligned16(S0)) || (choice && !aligned16(choice)) ||
      (logq && !aligned16(logq)) || (score && !aligned16(score)) ||
      (rescored && !aligned16(rescored)) || (CERT && (!aligned16(E) || !aligned16(packed_w))))
    return LILICORR_ERR_ALIGNMENT;
  if (workspace_bytes < decode_workspace_bytes(N, B, K, EXACT, CERT)) return LILICORR_ERR_WORKSPACE;
  const TailPlan tail = tail_plan(B, K, d, EXACT, CERT, kPairWaves * kWave, 160 * 1024 - 16);
  const size_t sw_bytes = EXACT ? 0 : (size_t)kPairWaves * K * K * 4;
  const size_t flag_off = ((sw_bytes > tail.bytes ? sw_bytes : tail.bytes) + 15) / 16 * 16;
  const size_t lds = flag_off + 16;
  if (lds > 160 * 1024) return LILICORR_ERR_UNSUPPORTED;
  const int nmat = (int)(B - 1) + (anchor_out ? 1 : 0);
  const dim3 grid((unsigned)(nmat > 0 ? (nmat + kPairWaves - 1) / kPairWaves : 1), (unsigned)N);
  unsigned char* ws = static_cast<unsigned char*>(workspace);
  uint32_t* counters = reinterpret_cast<uint32_t*>(ws);
  void* exchange = ws + counter_bytes(N);
  uint64_t* cmask = CERT ? static_cast<uint64_t*>(exchange) + N * tail.rows : nullptr;
  const uint16_t* e16 = CERT ? static_cast<const uint16_t*>(E) : nullptr;
  const float* w32 =
      CERT ? reinterpret_cast<const float*>(static_cast<const unsigned char*>(packed_w) +
                                            frag_bytes(d))
           : nullptr;
  auto go = [&](auto launch) {
    launch(grid, lds, stream, in_vec, out_vec, anchor_out, logp, ids, e16, V, B, K, d, sigma,
           logp_weight, margin, w32, tail, flag_off, S, S0, draft, choice, logq, score, rescored,
           counters, exchange, cmask);
  };
  // 16-row blocks per side as in lilicorr_pair_scores; the chunk width (the same columns in the
  // same order, so the same S) is narrower at K > 32, where eight waves share the registers
  if (K <= 16)
    go(launch_pair_walk<1, 4, 16, EXACT, CERT>);
  else if (K <= 32)
    go(launch_pair_walk<2, 2, 32, EXACT, CERT>);
  else
    go(launch_pair_walk<4, 1, 64, EXACT, CERT>);
  return launch_status();
}

}  // namespace
}  // namespace lilicorr

using namespace lilicorr;

extern "C" lilicorr_status lilicorr_pair_scores(const float* in_vec, const float* out_vec,
                                                const float* anchor_out, int64_t N, int64_t B,
                                                int K, int d, float sigma, float* S, float* S0,
                                                hipStream_t stream) {
  if (!in_vec || !out_vec) return LILICORR_ERR_INVALID_ARG;
  if (N < 1 || B < 1 || K < 1 || d < 1) return LILICORR_ERR_INVALID_ARG;
  if (B > 1 && !S) return LILICORR_ERR_INVALID_ARG;
  if (anchor_out && !S0) return LILICORR_ERR_INVALID_ARG;
  if (!isfinite(sigma)) return LILICORR_ERR_INVALID_ARG;
  if (K > 64 || d % 16 != 0 || d > 1024) return LILICORR_ERR_UNSUPPORTED;
  if (N > 65535 || B > 0x7fffffffll - 1) return LILICORR_ERR_UNSUPPORTED;
  if (!aligned16(in_vec) || !aligned16(out_vec) || (anchor_out && !aligned16(anchor_out)) ||
      (S && !aligned16(S)) || (S0 && !aligned16(S0)))
    return LILICORR_ERR_ALIGNMENT;
  const int npairs = (int)(B - 1) + (anchor_out ? 1 : 0);
  if (npairs == 0) return LILICORR_OK;
  const dim3 grid((unsigned)npairs, (unsigned)N);
  // 16-row blocks per side: ceil(K / 16); chunk width 64 columns at one block, 32 above (two
  // chunks of 32 columns keep a wave under 128 registers, so the stress shape's 3840 matrices
  // are all resident at once)
  if (K <= 16)
    launch_pairs<1, 4>(grid, stream, in_vec, out_vec, anchor_out, B, K, d, sigma, S, S0);
  else if (K <= 32)
    launch_pairs<2, 2>(grid, stream, in_vec, out_vec, anchor_out, B, K, d, sigma, S, S0);
  else
    launch_pairs<4, 2>(grid, stream, in_vec, out_vec, anchor_out, B, K, d, sigma, S, S0);
  return launch_status();
}

extern "C" lilicorr_status lilicorr_pair_walk(const float* in_vec, const float* out_vec,
                                              const float* anchor_out, const float* logp,
                                              const int32_t* ids, int64_t N, int64_t B, int K,
                                              int d, float sigma, float logp_weight, float* S,
                                              float* S0, int32_t* draft, int32_t* choice,
                                              float* logq, void* workspace, size_t workspace_bytes,
                                              hipStream_t stream) {
  return pairs_and_decode<false, false>(in_vec, out_vec, anchor_out, logp, ids, nullptr,
                                        LILICORR_BF16, 0, nullptr, N, B, K, d, sigma, logp_weight,
                                        0.f, S, S0, draft, choice, logq, nullptr, nullptr,
                                        workspace, workspace_bytes, stream);
}

extern "C" lilicorr_status lilicorr_pair_walk_certified(
    const float* in_vec, const float* out_vec, const float* anchor_out, const float* logp,
    const int32_t* ids, const void* E, lilicorr_dtype e_dtype, int64_t V, const void* packed_w,
    int64_t N, int64_t B, int K, int d, float sigma, float logp_weight, float margin, float* S,
    float* S0, int32_t* draft, int32_t* choice, float* logq, int32_t* rescored, void* workspace,
    size_t workspace_bytes, hipStream_t stream) {
  return pairs_and_decode<false, true>(in_vec, out_vec, anchor_out, logp, ids, E, e_dtype, V,
                                       packed_w, N, B, K, d, sigma, logp_weight, margin, S, S0,
                                       draft, choice, logq, nullptr, rescored, workspace,
                                       workspace_bytes, stream);
}

extern "C" lilicorr_status lilicorr_pair_viterbi(const float* in_vec, const float* out_vec,
                                                 const float* anchor_out, const float* logp,
                                                 const int32_t* ids, int64_t N, int64_t B, int K,
                                                 int d, float sigma, float logp_weight, float* S,
                                                 float* S0, int32_t* draft, int32_t* choice,
                                                 float* logq, float* score, void* workspace,
                                                 size_t workspace_bytes, hipStream_t stream) {
  return pairs_and_decode<true, false>(in_vec, out_vec, anchor_out, logp, ids, nullptr,
                                       LILICORR_BF16, 0, nullptr, N, B, K, d, sigma, logp_weight,
                                       0.f, S, S0, draft, choice, logq, score, nullptr, workspace,
                                       workspace_bytes, stream);
}
