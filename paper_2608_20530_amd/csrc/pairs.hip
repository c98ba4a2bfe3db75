// Step 3 of the path: batched pair matching scores, Eq. (pair):
//   S[n][t][k][k'] = sigma * cos(out[n][t][k], in[n][t+1][k'])
// one K x K matrix per adjacent slot pair, batched over the block (Sec. 3.5), and the anchor pair
// S0[n][k'] = sigma * cos(anchor_out[n], in[n][0][k']).
//
// One workgroup per (request, pair). The K left (out) and K right (in) vectors are streamed
// through LDS in 128-wide slices of the vector dimension, so each input vector is read from HBM
// exactly once; every thread accumulates dot products for a 2 x 2 block of (k, k') outputs and the
// squared norms are accumulated in the same pass.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "common.hpp"
#include "lilicorr.h"

namespace lilicorr {
namespace {

constexpr int kPairThreads = 256;
constexpr int kSlice = 128;
constexpr int kPad = kSlice + 4;  // row stride in LDS (floats), keeps 16-byte alignment

__global__ __launch_bounds__(kPairThreads) void pair_scores_kernel(
    const float* __restrict__ in_vec, const float* __restrict__ out_vec,
    const float* __restrict__ anchor_out, int64_t B, int K, int d, float sigma,
    float* __restrict__ S, float* __restrict__ S0) {
  __shared__ float lo[64 * kPad];  // left vectors (out of slot t, or the anchor)
  __shared__ float ro[64 * kPad];  // right vectors (in of slot t+1)
  __shared__ float nl[64], nr[64];

  const int64_t n = blockIdx.y;
  const int pair = blockIdx.x;  // 0..B-2 slot pairs, B-1 = anchor pair
  const bool anchor = pair == (int)(B - 1);
  const int KL = anchor ? 1 : K;
  const float* left = anchor ? anchor_out + n * d : out_vec + ((n * B + pair) * K) * (int64_t)d;
  const float* right = in_vec + ((n * B + (anchor ? 0 : pair + 1)) * K) * (int64_t)d;

  // output blocks of 2 x 2 (k, k') per thread
  const int KB = (K + 1) / 2;
  const int KLB = (KL + 1) / 2;
  const int nblk = KLB * KB;
  float acc[4][4];  // up to 4 blocks per thread (K <= 64 -> 32*32 blocks / 256 threads)
#pragma unroll
  for (int b = 0; b < 4; ++b)
#pragma unroll
    for (int q = 0; q < 4; ++q) acc[b][q] = 0.f;
  float nsq_l = 0.f, nsq_r = 0.f;  // thread tid < KL (left) / tid < K (right) owns a norm

  for (int base = 0; base < d; base += kSlice) {
    const int w = d - base < kSlice ? d - base : kSlice;  // multiple of 16
    const int w4 = w / 4;
    __syncthreads();
    for (int i = threadIdx.x; i < KL * w4; i += kPairThreads) {
      int r = i / w4, c = i % w4;
      *reinterpret_cast<float4*>(&lo[r * kPad + 4 * c]) =
          *reinterpret_cast<const float4*>(left + (int64_t)r * d + base + 4 * c);
    }
    for (int i = threadIdx.x; i < K * w4; i += kPairThreads) {
      int r = i / w4, c = i % w4;
      *reinterpret_cast<float4*>(&ro[r * kPad + 4 * c]) =
          *reinterpret_cast<const float4*>(right + (int64_t)r * d + base + 4 * c);
    }
    __syncthreads();
    if ((int)threadIdx.x < KL)
      for (int j = 0; j < w; ++j) nsq_l = fmaf(lo[threadIdx.x * kPad + j], lo[threadIdx.x * kPad + j], nsq_l);
    if ((int)threadIdx.x >= 64 && (int)threadIdx.x - 64 < K) {
      const int r = threadIdx.x - 64;
      for (int j = 0; j < w; ++j) nsq_r = fmaf(ro[r * kPad + j], ro[r * kPad + j], nsq_r);
    }
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      const int blk = threadIdx.x + b * kPairThreads;
      if (blk < nblk) {
        const int bi = blk / KB, bj = blk % KB;
        const int k0 = 2 * bi, k1 = k0 + 1 < KL ? k0 + 1 : k0;
        const int j0 = 2 * bj, j1 = j0 + 1 < K ? j0 + 1 : j0;
        const float* a0 = &lo[k0 * kPad];
        const float* a1 = &lo[k1 * kPad];
        const float* c0 = &ro[j0 * kPad];
        const float* c1 = &ro[j1 * kPad];
        float s00 = acc[b][0], s01 = acc[b][1], s10 = acc[b][2], s11 = acc[b][3];
        for (int j = 0; j < w; j += 4) {
          float4 x0 = *reinterpret_cast<const float4*>(a0 + j);
          float4 x1 = *reinterpret_cast<const float4*>(a1 + j);
          float4 y0 = *reinterpret_cast<const float4*>(c0 + j);
          float4 y1 = *reinterpret_cast<const float4*>(c1 + j);
          s00 = fmaf(x0.x, y0.x, s00); s00 = fmaf(x0.y, y0.y, s00); s00 = fmaf(x0.z, y0.z, s00); s00 = fmaf(x0.w, y0.w, s00);
          s01 = fmaf(x0.x, y1.x, s01); s01 = fmaf(x0.y, y1.y, s01); s01 = fmaf(x0.z, y1.z, s01); s01 = fmaf(x0.w, y1.w, s01);
          s10 = fmaf(x1.x, y0.x, s10); s10 = fmaf(x1.y, y0.y, s10); s10 = fmaf(x1.z, y0.z, s10); s10 = fmaf(x1.w, y0.w, s10);
          s11 = fmaf(x1.x, y1.x, s11); s11 = fmaf(x1.y, y1.y, s11); s11 = fmaf(x1.z, y1.z, s11); s11 = fmaf(x1.w, y1.w, s11);
        }
        acc[b][0] = s00; acc[b][1] = s01; acc[b][2] = s10; acc[b][3] = s11;
      }
    }
  }
  if ((int)threadIdx.x < KL) nl[threadIdx.x] = nsq_l;
  if ((int)threadIdx.x >= 64 && (int)threadIdx.x - 64 < K) nr[threadIdx.x - 64] = nsq_r;
  __syncthreads();
#pragma unroll
  for (int b = 0; b < 4; ++b) {
    const int blk = threadIdx.x + b * kPairThreads;
    if (blk < nblk) {
      const int bi = blk / KB, bj = blk % KB;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int k = 2 * bi + (q >> 1), kk = 2 * bj + (q & 1);
        if (k < KL && kk < K) {
          const float den = sqrtf(nl[k]) * sqrtf(nr[kk]);
          const float v = den > 0.f ? sigma * (acc[b][q] / den) : 0.f;
          if (anchor)
            S0[n * K + kk] = v;
          else
            S[((n * (B - 1) + pair) * K + k) * (int64_t)K + kk] = v;
        }
      }
    }
  }
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
  hipLaunchKernelGGL(pair_scores_kernel, dim3((unsigned)npairs, (unsigned)N), dim3(kPairThreads),
                     0, stream, in_vec, out_vec, anchor_out, B, K, d, sigma, S, S0);
  return launch_status();
}
