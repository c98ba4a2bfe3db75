// Step 3 of the path: batched pair matching scores, Eq. (pair):
//   S[n][t][k][k'] = sigma * cos(out[n][t][k], in[n][t+1][k'])
// one K x K matrix per adjacent slot pair, batched over the block (Sec. 3.5), and the anchor pair
// S0[n][k'] = sigma * cos(anchor_out[n], in[n][0][k']).
//
// One wavefront per (request, pair) matrix. The K left (out) and K right (in) vectors stream
// through LDS in 128-wide slices of the vector dimension, so every input vector is read from HBM
// exactly once. The 64 lanes form an 8 x 8 grid; lane (r, c) accumulates the dot products of left
// rows r, r+8, ... with right rows c, c+8, ... (a register block of up to 8 x 8), so each LDS read
// feeds several FMAs. The squared norms of the slice are accumulated one vector per lane.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "common.hpp"
#include "lilicorr.h"

namespace lilicorr {
namespace {

constexpr int kSlice = 128;
constexpr int kPad = kSlice + 4;  // LDS row stride in floats (16-byte aligned, spreads banks)

template <int R, int C>
__global__ __launch_bounds__(kWave) void pair_scores_kernel(
    const float* __restrict__ in_vec, const float* __restrict__ out_vec,
    const float* __restrict__ anchor_out, int64_t B, int K, int d, float sigma,
    float* __restrict__ S, float* __restrict__ S0) {
  __shared__ __attribute__((aligned(16))) float lo[8 * R * kPad];  // left vectors
  __shared__ __attribute__((aligned(16))) float ro[8 * C * kPad];  // right vectors
  __shared__ float nl[8 * R], nr[8 * C];

  const int lane = lane_id();
  const int64_t n = blockIdx.y;
  const int pair = blockIdx.x;  // 0..B-2 slot pairs; B-1 is the anchor pair when given
  const bool anchor = pair == (int)(B - 1);
  const int KL = anchor ? 1 : K;
  const float* left = anchor ? anchor_out + n * d : out_vec + ((n * B + pair) * K) * (int64_t)d;
  const float* right = in_vec + ((n * B + (anchor ? 0 : pair + 1)) * K) * (int64_t)d;
  const int lr = lane >> 3, lc = lane & 7;

  float acc[R][C];
#pragma unroll
  for (int i = 0; i < R; ++i)
#pragma unroll
    for (int j = 0; j < C; ++j) acc[i][j] = 0.f;
  float nsq = 0.f;   // lane v < KL: squared norm of left vector v
  float nsq2 = 0.f;  // lane v < K: squared norm of right vector v

  for (int base = 0; base < d; base += kSlice) {
    const int w = d - base < kSlice ? d - base : kSlice;  // a multiple of 16
    const int w4 = w >> 2;
    __syncthreads();
    // stage the slice: left rows then right rows, eight 16-byte loads in flight per lane
    {
      const int nl4 = KL * w4, n4 = (KL + K) * w4;
      for (int i0 = lane; i0 < n4; i0 += 8 * kWave) {
        float4 v[8];
#pragma unroll
        for (int b = 0; b < 8; ++b) {
          const int i = i0 + b * kWave;
          if (i < n4) {
            const bool l = i < nl4;
            const int ii = l ? i : i - nl4;
            const int r = ii / w4, c = ii - r * w4;
            v[b] = *reinterpret_cast<const float4*>((l ? left : right) + (int64_t)r * d + base + 4 * c);
          }
        }
#pragma unroll
        for (int b = 0; b < 8; ++b) {
          const int i = i0 + b * kWave;
          if (i < n4) {
            const bool l = i < nl4;
            const int ii = l ? i : i - nl4;
            const int r = ii / w4, c = ii - r * w4;
            *reinterpret_cast<float4*>(&(l ? lo : ro)[r * kPad + 4 * c]) = v[b];
          }
        }
      }
    }
    __syncthreads();
    // squared norms: lane v owns left vector v (v < KL); lane v also owns right vector v (v < K)
    if (lane < KL)
      for (int j = 0; j < w; j += 4) {
        const float4 a = *reinterpret_cast<const float4*>(&lo[lane * kPad + j]);
        nsq = fmaf(a.x, a.x, nsq); nsq = fmaf(a.y, a.y, nsq);
        nsq = fmaf(a.z, a.z, nsq); nsq = fmaf(a.w, a.w, nsq);
      }
    if (lane < K)
      for (int j = 0; j < w; j += 4) {
        const float4 a = *reinterpret_cast<const float4*>(&ro[lane * kPad + j]);
        nsq2 = fmaf(a.x, a.x, nsq2); nsq2 = fmaf(a.y, a.y, nsq2);
        nsq2 = fmaf(a.z, a.z, nsq2); nsq2 = fmaf(a.w, a.w, nsq2);
      }
    for (int j = 0; j < w; j += 4) {
      float4 a[R], b[C];
#pragma unroll
      for (int i = 0; i < R; ++i) a[i] = *reinterpret_cast<const float4*>(&lo[(lr + 8 * i) * kPad + j]);
#pragma unroll
      for (int q = 0; q < C; ++q) b[q] = *reinterpret_cast<const float4*>(&ro[(lc + 8 * q) * kPad + j]);
#pragma unroll
      for (int i = 0; i < R; ++i)
#pragma unroll
        for (int q = 0; q < C; ++q) {
          float s = acc[i][q];
          s = fmaf(a[i].x, b[q].x, s);
          s = fmaf(a[i].y, b[q].y, s);
          s = fmaf(a[i].z, b[q].z, s);
          s = fmaf(a[i].w, b[q].w, s);
          acc[i][q] = s;
        }
    }
  }
  if (lane < KL) nl[lane] = nsq;
  if (lane < K) nr[lane] = nsq2;
  __syncthreads();
#pragma unroll
  for (int i = 0; i < R; ++i)
#pragma unroll
    for (int q = 0; q < C; ++q) {
      const int k = lr + 8 * i, kk = lc + 8 * q;
      if (k < KL && kk < K) {
        const float den = sqrtf(nl[k]) * sqrtf(nr[kk]);
        const float v = den > 0.f ? sigma * (acc[i][q] / den) : 0.f;
        if (anchor)
          S0[n * K + kk] = v;
        else
          S[((n * (B - 1) + pair) * K + k) * (int64_t)K + kk] = v;
      }
    }
}

template <int R, int C>
void launch_pairs(dim3 grid, hipStream_t stream, const float* in_vec, const float* out_vec,
                  const float* anchor_out, int64_t B, int K, int d, float sigma, float* S,
                  float* S0) {
  hipLaunchKernelGGL((pair_scores_kernel<R, C>), grid, dim3(kWave), 0, stream, in_vec, out_vec,
                     anchor_out, B, K, d, sigma, S, S0);
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
  // register block per lane: ceil(K / 8) rows x ceil(K / 8) columns
  if (K <= 8)
    launch_pairs<1, 1>(grid, stream, in_vec, out_vec, anchor_out, B, K, d, sigma, S, S0);
  else if (K <= 16)
    launch_pairs<2, 2>(grid, stream, in_vec, out_vec, anchor_out, B, K, d, sigma, S, S0);
  else if (K <= 32)
    launch_pairs<4, 4>(grid, stream, in_vec, out_vec, anchor_out, B, K, d, sigma, S, S0);
  else
    launch_pairs<8, 8>(grid, stream, in_vec, out_vec, anchor_out, B, K, d, sigma, S, S0);
  return launch_status();
}
