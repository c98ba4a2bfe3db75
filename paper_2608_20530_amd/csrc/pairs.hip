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
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "common.hpp"
#include "lilicorr.h"

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

template <int NBL, int NBR, int S4>
__global__ __launch_bounds__(kWave) void pair_scores_kernel(
    const float* __restrict__ in_vec, const float* __restrict__ out_vec,
    const float* __restrict__ anchor_out, int64_t B, int K, int d, float sigma,
    float* __restrict__ S, float* __restrict__ S0) {
  constexpr int kCols = 16 * S4;  // columns per chunk
  const int lane = lane_id();
  const int r = lane & 15, q = lane >> 4;
  const int64_t n = blockIdx.y;
  const int pair = blockIdx.x;  // 0..B-2 slot pairs; B-1 is the anchor pair when given
  const bool anchor = pair == (int)(B - 1);
  const int KL = anchor ? 1 : K;
  const float* left = anchor ? anchor_out + n * d : out_vec + ((n * B + pair) * K) * (int64_t)d;
  const float* right = in_vec + ((n * B + (anchor ? 0 : pair + 1)) * K) * (int64_t)d;
  const __amdgpu_buffer_rsrc_t rl = rows_rsrc(left, KL, d), rr = rows_rsrc(right, K, d);

  f32x4 acc[NBL][NBR];
#pragma unroll
  for (int bl = 0; bl < NBL; ++bl)
#pragma unroll
    for (int br = 0; br < NBR; ++br) acc[bl][br] = f32x4{0.f, 0.f, 0.f, 0.f};
  float nl[NBL], nr[NBR];  // squared norms of this lane's share of left / right row r
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

  // lane l holds tile entries (row 4(l/16) + i, column l % 16), i = 0..3
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
          const float v = den > 0.f ? sigma * (acc[bl][br][i] / den) : 0.f;
          if (anchor)
            S0[n * K + kk] = v;
          else
            S[((n * (B - 1) + pair) * K + k) * (int64_t)K + kk] = v;
        }
      }
    }
}

template <int NB, int S4>
void launch_pairs(dim3 grid, hipStream_t stream, const float* in_vec, const float* out_vec,
                  const float* anchor_out, int64_t B, int K, int d, float sigma, float* S,
                  float* S0) {
  hipLaunchKernelGGL((pair_scores_kernel<NB, NB, S4>), grid, dim3(kWave), 0, stream, in_vec,
                     out_vec, anchor_out, B, K, d, sigma, S, S0);
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
