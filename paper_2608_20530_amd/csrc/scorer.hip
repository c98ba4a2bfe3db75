// Scoring-Transformer stand-in on gfx950: the encoder of the paper's speculative head
// (implementation appendix, "Architecture"; widths and depth from the hyper-parameter table), a
// stack of pre-norm bidirectional Transformer layers over each request's candidate lattice of
// S slots x K candidates, with per-head slot-distance and same-slot attention biases.
//
// One layer is seven launches:
//   rmsnorm -> bf16            X fp32 [M][H] -> xn bf16                       (HBM bound)
//   GEMM  xn . Wqkv            -> Q, K bf16 [M][2H] and V^T bf16 [N][H][Lv]   (matrix cores)
//   lattice attention          one workgroup per (request, head); K and V^T of the request in LDS
//   GEMM  attn . Wo, X +=      residual update in place                      (matrix cores)
//   rmsnorm -> bf16
//   GEMM  hn . W1 -> silu -> bf16 [M][F]                                     (matrix cores)
//   GEMM  a . W2, X +=                                                        (matrix cores)
// M = N * L token rows. Every matrix-core input is bf16 (round to nearest even), products
// accumulate in fp32 on v_mfma_f32_16x16x32_bf16, the residual stream stays fp32.
//
// GEMM: C[M][N] = A[M][K] . B[K][N] with B stored transposed (Bt[N][K], written once by the pack
// call) so both operands stream K-contiguous 16-byte chunks. A 128 x 128 tile per workgroup of
// four waves (2 x 2, 64 x 64 each, 16 accumulator tiles per wave), 64-deep k-stages double-
// buffered in LDS with an XOR swizzle of the 16-byte chunks (row r's chunk c at c ^ (r & 7)),
// the next stage's global loads in flight while the current stage's MFMAs run. Rows past M read
// zeros through the buffer descriptor's range check and are not stored.
//
// Attention: S^T = K Q^T per 16-query chunk (keys are the MFMA rows), so each lane ends up with
// one query's logits over keys 16t + 4g + i (g = lane / 16); the softmax reduces over tiles in
// registers and over the four lane groups by shuffles, and the probabilities are already in the
// A-operand layout of P V once the k slots of a 32-key step are read as keys (4g + j, 16 + 4g + j):
// V^T is read with the same key order, so no LDS round trip is needed for P.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "common.hpp"
#include "lilicorr.h"

namespace lilicorr {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
typedef int i32x4 __attribute__((ext_vector_type(4)));

constexpr int kHd = 128;  // head width
constexpr float kEps = 1e-6f;
constexpr float kLog2e = 1.4426950408889634f;
constexpr int kBK = 64;
constexpr int kGemmThreads = 256;
constexpr int kGroup = 8;  // row blocks per tile group (L2 blocking of the GEMM grid)
constexpr int kAttnThreads = 512;
constexpr int kMaxL = 256;
constexpr int kMaxH = 4096;
constexpr int kMaxF = 16384;
constexpr int64_t kMaxS = 256;
constexpr size_t kAlign = 256;

inline size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

// fp32 -> bf16, round to nearest even: one v_cvt_pk_bf16_f32 per pair of values on gfx950
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2{lo, hi}), bf16x2));
}

__device__ __forceinline__ uint32_t bf16_rne(float x) {
  return __builtin_bit_cast(uint16_t, (__bf16)x);
}

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, 0x00020000);
}

// ---- RMSNorm -> bf16 ----------------------------------------------------------------------------
// One wave per row of H = NV * 256 fp32 values: y = bf16(x / sqrt(mean(x^2) + eps) * g).
template <int NV>
__global__ __launch_bounds__(256) void rmsnorm_bf16_kernel(const float* __restrict__ X,
                                                           const float* __restrict__ g,
                                                           uint16_t* __restrict__ Y, int64_t M) {
  constexpr int H = NV * 256;
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= M) return;
  const float4* x = reinterpret_cast<const float4*>(X + row * H);
  float4 v[NV];
  float ss = 0.f;
#pragma unroll
  for (int j = 0; j < NV; ++j) {
    v[j] = x[j * 64 + lane];
    ss += v[j].x * v[j].x + v[j].y * v[j].y + v[j].z * v[j].z + v[j].w * v[j].w;
  }
  ss = wave_sum(ss);
  const float inv = 1.0f / sqrtf(ss / (float)H + kEps);
  const float4* gg = reinterpret_cast<const float4*>(g);
  u32x2* y = reinterpret_cast<u32x2*>(Y + row * H);
#pragma unroll
  for (int j = 0; j < NV; ++j) {
    const float4 w = gg[j * 64 + lane];
    y[j * 64 + lane] = u32x2{pack_bf16x2(v[j].x * inv * w.x, v[j].y * inv * w.y),
                             pack_bf16x2(v[j].z * inv * w.z, v[j].w * inv * w.w)};
  }
}

// ---- GEMM on the bf16 matrix cores ------------------------------------------------------------
enum { kModeQKV = 0, kModeResid = 1, kModeSilu = 2 };

struct GemmArgs {
  const uint16_t* A;   // [M][K] bf16
  const uint16_t* Bt;  // [N][K] bf16 (B transposed)
  int64_t M;
  int K, N;
  float* X;      // resid: X[M][N] += A . B
  uint16_t* Y;   // silu: Y[M][N] = bf16(silu(A . B)); qkv: Q and K columns, Y[M][2H]
  uint16_t* Vt;  // qkv: V columns transposed per request, Vt[M / L][H][Lv]
  int H, L, Lv;
};

// One workgroup of four waves (2 x 2) computes a (32 WTM) x (32 WTN) tile; each wave a
// (16 WTM) x (16 WTN) block of WTM x WTN accumulator tiles.
template <int MODE, int WTM, int WTN>
__global__ __launch_bounds__(kGemmThreads) void gemm_bf16_kernel(GemmArgs p) {
  constexpr int BM = 32 * WTM, BN = 32 * WTN;
  constexpr int CA = BM * 8 / kGemmThreads, CB = BN * 8 / kGemmThreads;  // chunks per thread
  extern __shared__ __attribute__((aligned(16))) unsigned char gemm_smem[];
  uint16_t* sA = reinterpret_cast<uint16_t*>(gemm_smem);   // [2][BM * kBK]
  uint16_t* sB = sA + 2 * BM * kBK;                        // [2][BN * kBK]
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int ntn = p.N / BN;
  // Workgroups are dealt to the eight XCDs round robin; when the grid divides evenly, each XCD
  // takes a contiguous run of tile numbers. Tile numbers run over groups of kGroup row blocks,
  // column blocks outer, so the workgroups an XCD holds at once share A rows and B columns in
  // its L2.
  const uint32_t nt = gridDim.x;
  const uint32_t t = (nt % 8u == 0u) ? (blockIdx.x % 8u) * (nt / 8u) + blockIdx.x / 8u
                                     : blockIdx.x;
  const int64_t ntm = (p.M + BM - 1) / BM;
  const int64_t per_group = (int64_t)kGroup * ntn;
  const int64_t grp = t / per_group;
  const int64_t rows_in = (ntm - grp * kGroup) < kGroup ? (ntm - grp * kGroup) : kGroup;
  const int64_t r = t - grp * per_group;
  const int64_t tm = grp * kGroup + r % rows_in;
  const int tn = (int)(r / rows_in);
  const int64_t m0 = tm * BM;
  const int n0 = tn * BN;
  const uint32_t K2 = (uint32_t)p.K * 2u;
  const __amdgpu_buffer_rsrc_t ra = make_rsrc(p.A, (uint32_t)p.M * K2);
  const __amdgpu_buffer_rsrc_t rb = make_rsrc(p.Bt, (uint32_t)p.N * K2);

  // staging: thread tid moves chunks tid + 256 j of each tile; chunk c is row c / 8, 16-byte
  // column c % 8, stored at column (c % 8) ^ (row % 8)
  uint32_t offA[CA], offB[CB];
  int ldsA[CA], ldsB[CB];
#pragma unroll
  for (int j = 0; j < CA; ++j) {
    const int c = tid + j * kGemmThreads;
    const int row = c >> 3, kc = c & 7;
    offA[j] = (uint32_t)(m0 + row) * K2 + (uint32_t)kc * 16u;
    ldsA[j] = row * kBK + ((kc ^ (row & 7)) << 3);
  }
#pragma unroll
  for (int j = 0; j < CB; ++j) {
    const int c = tid + j * kGemmThreads;
    const int row = c >> 3, kc = c & 7;
    offB[j] = (uint32_t)(n0 + row) * K2 + (uint32_t)kc * 16u;
    ldsB[j] = row * kBK + ((kc ^ (row & 7)) << 3);
  }
  // two register sets: the loads of stage s + 2 are issued while stage s is multiplied, and
  // stored to LDS only at the end of stage s + 1
  u32x4 g0[CA + CB], g1[WTM * WTN > 16 ? 1 : CA + CB];
  auto gload = [&](u32x4 (&g)[CA + CB], int k0) {
    const uint32_t kb = (uint32_t)k0 * 2u;
#pragma unroll
    for (int j = 0; j < CA; ++j)
      g[j] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(ra, offA[j] + kb, 0, 0));
#pragma unroll
    for (int j = 0; j < CB; ++j)
      g[CA + j] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rb, offB[j] + kb, 0, 0));
  };
  auto lstore = [&](const u32x4 (&g)[CA + CB], int buf) {
#pragma unroll
    for (int j = 0; j < CA; ++j) *reinterpret_cast<u32x4*>(&sA[buf * BM * kBK + ldsA[j]]) = g[j];
#pragma unroll
    for (int j = 0; j < CB; ++j) *reinterpret_cast<u32x4*>(&sB[buf * BN * kBK + ldsB[j]]) = g[CA + j];
  };

  // fragment reads: row (lane & 15) of each 16-row block, k chunk ks * 4 + lane / 16
  int rowA[WTM], rowB[WTN], sw[2];
#pragma unroll
  for (int i = 0; i < WTM; ++i) rowA[i] = (wm * 16 * WTM + i * 16 + (lane & 15)) * kBK;
#pragma unroll
  for (int i = 0; i < WTN; ++i) rowB[i] = (wn * 16 * WTN + i * 16 + (lane & 15)) * kBK;
#pragma unroll
  for (int ks = 0; ks < 2; ++ks) sw[ks] = ((ks * 4 + (lane >> 4)) ^ (lane & 7)) << 3;

  f32x4 acc[WTM][WTN];
#pragma unroll
  for (int i = 0; i < WTM; ++i)
#pragma unroll
    for (int j = 0; j < WTN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  auto multiply = [&](int buf) {
    const uint16_t* as = sA + buf * BM * kBK;
    const uint16_t* bs = sB + buf * BN * kBK;
    // both k halves' fragments are read before the first MFMA, so the second half's reads are
    // in flight while the first half's MFMAs issue
    bf16x8 a[2][WTM], b[2][WTN];
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
#pragma unroll
      for (int i = 0; i < WTM; ++i)
        a[ks][i] = *reinterpret_cast<const bf16x8*>(as + rowA[i] + sw[ks]);
#pragma unroll
      for (int j = 0; j < WTN; ++j)
        b[ks][j] = *reinterpret_cast<const bf16x8*>(bs + rowB[j] + sw[ks]);
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int ks = 0; ks < 2; ++ks)
#pragma unroll
      for (int i = 0; i < WTM; ++i)
#pragma unroll
        for (int j = 0; j < WTN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[ks][i], b[ks][j], acc[i][j], 0, 0, 0);
  };
  // Stage s sits in LDS buffer s % 2 and, until stored, in register set s % 2. The loads and
  // stores are unconditional (the last two steps reload the final stage and store into the
  // buffer nobody reads again): behind a branch, the compiler could no longer tell which loads
  // are still in flight at the stores and would wait for all of them. The scheduling barriers
  // keep the loads at the head of the step, ahead of the MFMAs (left alone, the scheduler sinks
  // them below the MFMAs to save registers).
  auto step = [&](auto& cur, auto& nxt, int s, int nk) {
    gload(cur, (s + 2 < nk ? s + 2 : nk - 1) * kBK);
    __builtin_amdgcn_sched_barrier(0);
    multiply(s & 1);
    __builtin_amdgcn_sched_barrier(0);
    lstore(nxt, (s + 1) & 1);
    __syncthreads();
  };
  const int nk = p.K / kBK;  // even: K is a multiple of 128
  if constexpr (WTM * WTN > 16) {
    // large wave tiles: one register set, loaded one stage ahead (a stage's 2 * WTM * WTN MFMAs
    // cover the load latency), which keeps the accumulators and fragments in registers
    auto step1 = [&](int s) {
      gload(g0, (s + 1 < nk ? s + 1 : nk - 1) * kBK);
      __builtin_amdgcn_sched_barrier(0);
      multiply(s & 1);
      __builtin_amdgcn_sched_barrier(0);
      lstore(g0, (s + 1) & 1);
      __syncthreads();
    };
    gload(g0, 0);
    lstore(g0, 0);
    __syncthreads();
    for (int s = 0; s < nk; ++s) step1(s);
  } else {
    gload(g0, 0);
    gload(g1, kBK);
    lstore(g0, 0);
    __syncthreads();
    for (int s = 0; s < nk; s += 2) {
      step(g0, g1, s, nk);
      step(g1, g0, s + 1, nk);
    }
  }

  // epilogue: lane holds rows 4 * (lane / 16) + j of each 16-row block, column lane % 16
  const int64_t rbase = m0 + wm * 16 * WTM + 4 * (lane >> 4);
  const int cbase = n0 + wn * 16 * WTN + (lane & 15);
  const bool vpart = MODE == kModeQKV && n0 >= 2 * p.H;  // uniform: a tile is all Q/K or all V
#pragma unroll
  for (int mt = 0; mt < WTM; ++mt) {
    // request and lattice position of the block's first row (rows < 2^31), then stepped
    const int64_t row0 = rbase + mt * 16;
    int rq = 0, l = 0;
    if (vpart) {
      rq = (int)row0 / p.L;
      l = (int)row0 - rq * p.L;
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int64_t row = row0 + j;
      if (row < p.M) {
#pragma unroll
        for (int nt2 = 0; nt2 < WTN; ++nt2) {
          const int col = cbase + nt2 * 16;
          const float v = acc[mt][nt2][j];
          if constexpr (MODE == kModeResid) {
            float* x = p.X + row * p.N + col;
            *x = *x + v;
          } else if constexpr (MODE == kModeSilu) {
            // silu(v) = v / (1 + e^-v), the reciprocal on the hardware unit (the result is
            // rounded to bf16 next)
            p.Y[row * p.N + col] =
                (uint16_t)bf16_rne(v * __builtin_amdgcn_rcpf(1.0f + __expf(-v)));
          } else {
            if (!vpart)
              p.Y[row * (2 * p.H) + col] = (uint16_t)bf16_rne(v);
            else
              p.Vt[((int64_t)rq * p.H + (col - 2 * p.H)) * p.Lv + l] = (uint16_t)bf16_rne(v);
          }
        }
      }
      if (vpart && ++l == p.L) {
        l = 0;
        ++rq;
      }
    }
  }
}

template <int MODE, int WTM, int WTN>
void launch_gemm_tile(const GemmArgs& a, hipStream_t stream) {
  constexpr int BM = 32 * WTM, BN = 32 * WTN;
  constexpr size_t lds = (size_t)2 * (BM + BN) * kBK * 2;
  static const hipError_t attr = hipFuncSetAttribute(
      reinterpret_cast<const void*>(gemm_bf16_kernel<MODE, WTM, WTN>),
      hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  (void)attr;
  const int64_t tiles = (a.M + BM - 1) / BM * (a.N / BN);
  hipLaunchKernelGGL((gemm_bf16_kernel<MODE, WTM, WTN>), dim3((unsigned)tiles),
                     dim3(kGemmThreads), lds, stream, a);
}

// 128 x 128 tiles (64 x 64 per wave): two workgroups per compute unit, so one's barrier waits
// and epilogue overlap the other's MFMAs (256 x 256 tiles at one wave per SIMD measured 1.3-4.6x
// slower)
// ---- 128 x 256 tiles, operands by DMA ---------------------------------------------------------
// Four waves (2 x 2), each a 64 x 128 block (32 accumulator tiles): a fragment read feeds 4 or 8
// MFMAs, 12 KB of LDS reads per 32 MFMAs instead of 8 KB per 16. The operands reach LDS by DMA
// (buffer loads with an LDS destination, lane i of a load writing 16 bytes at 16 i past the
// wave's base), in a ring of three 32-deep stages (72 KB, two workgroups per compute unit); a
// stage row is 64 bytes and chunk c of row r sits at position c ^ ((r / 2) % 4).
constexpr int kDBK = 32;
constexpr int kDA = 128 * kDBK, kDB = 256 * kDBK;  // elements of one stage of A, of B

typedef __attribute__((address_space(3))) void* lds_ptr_t;

template <int MODE>
__global__ __launch_bounds__(kGemmThreads, 2) void gemm_dma_kernel(GemmArgs p) {
  extern __shared__ __attribute__((aligned(16))) unsigned char dma_smem[];
  uint16_t* ring = reinterpret_cast<uint16_t*>(dma_smem);  // [3][A stage, B stage]
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int ntn = p.N / 256;
  const uint32_t nt = gridDim.x;
  const uint32_t t = (nt % 8u == 0u) ? (blockIdx.x % 8u) * (nt / 8u) + blockIdx.x / 8u
                                     : blockIdx.x;
  const int64_t ntm = (p.M + 127) / 128;
  const int64_t per_group = (int64_t)kGroup * ntn;
  const int64_t grp = t / per_group;
  const int64_t rows_in = (ntm - grp * kGroup) < kGroup ? (ntm - grp * kGroup) : kGroup;
  const int64_t r = t - grp * per_group;
  const int64_t m0 = (grp * kGroup + r % rows_in) * 128;
  const int n0 = (int)(r / rows_in) * 256;
  const uint32_t K2 = (uint32_t)p.K * 2u;
  const __amdgpu_buffer_rsrc_t ra = make_rsrc(p.A, (uint32_t)p.M * K2);
  const __amdgpu_buffer_rsrc_t rb = make_rsrc(p.Bt, (uint32_t)p.N * K2);
  // DMA slots: A has 512 (wave w: 128 w .. 128 w + 127, two loads), B 1024 (four loads)
  uint32_t offA[2], offB[4];
#pragma unroll
  for (int d = 0; d < 2; ++d) {
    const int q = wave * 128 + d * 64 + lane;
    const int row = q >> 2, kc = (q & 3) ^ ((row >> 1) & 3);
    offA[d] = (uint32_t)(m0 + row) * K2 + (uint32_t)kc * 16u;
  }
#pragma unroll
  for (int d = 0; d < 4; ++d) {
    const int q = wave * 256 + d * 64 + lane;
    const int row = q >> 2, kc = (q & 3) ^ ((row >> 1) & 3);
    offB[d] = (uint32_t)(n0 + row) * K2 + (uint32_t)kc * 16u;
  }
  auto dma = [&](int buf, int stage) {
    uint16_t* da = ring + buf * (kDA + kDB);
    uint16_t* db = da + kDA;
    const int soff = stage * kDBK * 2;
#pragma unroll
    for (int d = 0; d < 2; ++d)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          ra, (lds_ptr_t)(da + (wave * 128 + d * 64) * 8), 16, offA[d], soff, 0, 0);
#pragma unroll
    for (int d = 0; d < 4; ++d)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          rb, (lds_ptr_t)(db + (wave * 256 + d * 64) * 8), 16, offB[d], soff, 0, 0);
  };
  int rowA[4], rowB[8];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int x = wm * 64 + i * 16 + (lane & 15);
    rowA[i] = x * kDBK + (((lane >> 4) ^ ((x >> 1) & 3)) << 3);
  }
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int x = wn * 128 + i * 16 + (lane & 15);
    rowB[i] = x * kDBK + (((lane >> 4) ^ ((x >> 1) & 3)) << 3);
  }
  f32x4 acc[4][8];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  auto multiply = [&](int buf) {
    const uint16_t* as = ring + buf * (kDA + kDB);
    const uint16_t* bs = as + kDA;
    bf16x8 a[4], b[8];
#pragma unroll
    for (int i = 0; i < 4; ++i) a[i] = *reinterpret_cast<const bf16x8*>(as + rowA[i]);
#pragma unroll
    for (int j = 0; j < 8; ++j) b[j] = *reinterpret_cast<const bf16x8*>(bs + rowB[j]);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 8; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
  };
  // the bare s_barrier after the wave's own DMA wait (six loads per stage per wave: stage s + 1
  // has landed when only stage s + 2's six are in flight); __syncthreads() would add a release
  // fence waiting for every DMA
  const int nk = p.K / kDBK;  // a multiple of 4
  dma(0, 0);
  dma(1, 1);
  __asm__ volatile("s_waitcnt vmcnt(6)\n\ts_barrier" ::: "memory");
  int s = 0;
  for (; s + 3 <= nk; s += 3) {
#pragma unroll
    for (int u = 0; u < 3; ++u) {
      dma((u + 2) % 3, s + u + 2 < nk ? s + u + 2 : nk - 1);
      multiply(u);
      __asm__ volatile("s_waitcnt vmcnt(6)\n\ts_barrier" ::: "memory");
    }
  }
  for (int u = 0; s < nk; ++s, ++u) {
    dma((u + 2) % 3, s + 2 < nk ? s + 2 : nk - 1);
    multiply(u);
    __asm__ volatile("s_waitcnt vmcnt(6)\n\ts_barrier" ::: "memory");
  }
  __asm__ volatile("s_waitcnt vmcnt(0)" ::: "memory");

  // epilogue: lane holds rows 4 * (lane / 16) + j of each 16-row block, column lane % 16
  const int64_t rbase = m0 + wm * 64 + 4 * (lane >> 4);
  const int cbase = n0 + wn * 128 + (lane & 15);
  const bool vpart = MODE == kModeQKV && n0 >= 2 * p.H;
  // four consecutive rows of one request when L % 4 == 0 (a block's rows start at a multiple of
  // 4): one 8-byte store per column into V^T
  const bool vfast = vpart && (p.L % 4 == 0);
  if constexpr (MODE == kModeResid) {
    // X += acc: the 32 values of 16-row block mt + 1 are loaded (rows past M clamped to the last
    // row and not stored) before block mt is added and stored, so the loads of consecutive
    // blocks overlap instead of each block waiting on its own
    float xv[2][4][8];
    auto load = [&](int mt, float (&d)[4][8]) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        int64_t row = rbase + mt * 16 + j;
        row = row < p.M ? row : p.M - 1;
#pragma unroll
        for (int nt2 = 0; nt2 < 8; ++nt2) d[j][nt2] = p.X[row * p.N + cbase + nt2 * 16];
      }
    };
    load(0, xv[0]);
#pragma unroll
    for (int mt = 0; mt < 4; ++mt) {
      if (mt + 1 < 4) load(mt + 1, xv[(mt + 1) & 1]);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int64_t row = rbase + mt * 16 + j;
        if (row < p.M) {
#pragma unroll
          for (int nt2 = 0; nt2 < 8; ++nt2)
            p.X[row * p.N + cbase + nt2 * 16] = xv[mt & 1][j][nt2] + acc[mt][nt2][j];
        }
      }
    }
    return;
  }
#pragma unroll
  for (int mt = 0; mt < 4; ++mt) {
    const int64_t row0 = rbase + mt * 16;
    if (vfast) {
      if (row0 < p.M) {
        const int rq4 = (int)row0 / p.L, l4 = (int)row0 - rq4 * p.L;
#pragma unroll
        for (int nt2 = 0; nt2 < 8; ++nt2) {
          const int col = cbase + nt2 * 16;
          *reinterpret_cast<u32x2*>(p.Vt + ((int64_t)rq4 * p.H + (col - 2 * p.H)) * p.Lv + l4) =
              u32x2{pack_bf16x2(acc[mt][nt2][0], acc[mt][nt2][1]),
                    pack_bf16x2(acc[mt][nt2][2], acc[mt][nt2][3])};
        }
      }
      continue;
    }
    int rq = 0, l = 0;
    if (vpart) {
      rq = (int)row0 / p.L;
      l = (int)row0 - rq * p.L;
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int64_t row = row0 + j;
      if (row < p.M) {
#pragma unroll
        for (int nt2 = 0; nt2 < 8; ++nt2) {
          const int col = cbase + nt2 * 16;
          const float v = acc[mt][nt2][j];
          if constexpr (MODE == kModeResid) {
            float* x = p.X + row * p.N + col;
            *x = *x + v;
          } else if constexpr (MODE == kModeSilu) {
            p.Y[row * p.N + col] =
                (uint16_t)bf16_rne(v * __builtin_amdgcn_rcpf(1.0f + __expf(-v)));
          } else {
            if (!vpart)
              p.Y[row * (2 * p.H) + col] = (uint16_t)bf16_rne(v);
            else
              p.Vt[((int64_t)rq * p.H + (col - 2 * p.H)) * p.Lv + l] = (uint16_t)bf16_rne(v);
          }
        }
      }
      if (vpart && ++l == p.L) {
        l = 0;
        ++rq;
      }
    }
  }
}

template <int MODE>
void launch_gemm_dma(const GemmArgs& a, hipStream_t stream) {
  constexpr size_t lds = (size_t)3 * (kDA + kDB) * 2;
  static const hipError_t attr = hipFuncSetAttribute(
      reinterpret_cast<const void*>(gemm_dma_kernel<MODE>),
      hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  (void)attr;
  const int64_t tiles = (a.M + 127) / 128 * (a.N / 256);
  hipLaunchKernelGGL(gemm_dma_kernel<MODE>, dim3((unsigned)tiles), dim3(kGemmThreads), lds,
                     stream, a);
}

// 128 x 256 DMA-fed tiles when the output width allows, else 128 x 128
template <int MODE>
void launch_gemm(const GemmArgs& a, hipStream_t stream) {
  if (a.N % 256 == 0)
    launch_gemm_dma<MODE>(a, stream);
  else
    launch_gemm_tile<MODE, 4, 4>(a, stream);
}

// ---- lattice attention ----------------------------------------------------------------------
struct AttnArgs {
  const uint16_t* qk;    // [N * L][2H]: Q at column h * 128, K at H + h * 128
  const uint16_t* vt;    // [N][H][Lv]
  const float* dist;     // [heads][2S - 1]
  const float* same;     // [heads]
  uint16_t* out;         // [N * L][H]
  int S, K, L, Lv, Lp, H, heads;
};

// Lattices with S * Lp <= kBiasRows keep one row of additive logit bias per query slot in LDS
// (slot-distance and same-slot terms in log2 units, -inf past the last key); larger ones look the
// bias up per element.
constexpr int kBiasRows = 4096;

inline bool attn_bias_rows(int Lp, int S) { return (int64_t)S * Lp <= kBiasRows; }

inline size_t attn_lds_bytes(int Lp, int S) {
  return (size_t)Lp * kHd * 2 + (size_t)kHd * (Lp + 4) * 2 + (size_t)((2 * S + 3) & ~3) * 4 +
         (size_t)Lp * 4 + (attn_bias_rows(Lp, S) ? (size_t)S * Lp * 4 : 0);
}

// NT = Lp / 16 key tiles (even, 2..16): the key loops are unrolled exactly.
template <bool ROWS, int NT>
__global__ __launch_bounds__(kAttnThreads) void lattice_attention_kernel(AttnArgs p) {
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  const int n = blockIdx.x / p.heads, h = blockIdx.x - n * p.heads;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  constexpr int Lp = 16 * NT, vstride = Lp + 4;
  const int L = p.L;
  uint16_t* sK = reinterpret_cast<uint16_t*>(smem);        // [Lp][128], chunk c of key j at c ^ (j % 8)
  uint16_t* sV = sK + Lp * kHd;                              // [128][Lp + 4]
  float* sBias = reinterpret_cast<float*>(sV + kHd * vstride);  // [2S - 1] dist, [2S - 1] same (log2 units)
  int* sSlot = reinterpret_cast<int*>(sBias + ((2 * p.S + 3) & ~3));  // [Lp] key slot, -1 past L
  float* sRow = reinterpret_cast<float*>(sSlot + Lp);  // ROWS: [S][Lp] bias of query slot x key
  const int64_t tok0 = (int64_t)n * L;
  const int H2 = 2 * p.H;

  const int g = lane >> 4, c16 = lane & 15;
  const int nq = (L + 15) / 16;
  // Q fragments of this wave's first query chunk, loaded while K and V^T are staged
  bf16x8 qf[4];
  auto load_q = [&](int qc) {
    const int q = qc * 16 + c16;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      u32x4 v = u32x4{0u, 0u, 0u, 0u};
      if (q < L)
        v = *reinterpret_cast<const u32x4*>(p.qk + (tok0 + q) * H2 + h * kHd + ks * 32 + g * 8);
      qf[ks] = __builtin_bit_cast(bf16x8, v);
    }
  };
  if (wave < nq) load_q(wave);

  // K rows (16 chunks of 16 bytes each) and V^T rows (Lp / 8 = 2 NT chunks each): NT / 2 chunks
  // of each per thread, every load issued before the first LDS store
  constexpr int kPer = NT / 2;  // (Lp * 16) / 512 == (128 * Lp / 8) / 512
  constexpr int cpr = 2 * NT;
  u32x4 kv[2 * kPer];
#pragma unroll
  for (int b = 0; b < kPer; ++b) {
    const int i = tid + b * kAttnThreads;
    const int j = i >> 4, c = i & 15;
    kv[b] = u32x4{0u, 0u, 0u, 0u};
    if (j < L)
      kv[b] = *reinterpret_cast<const u32x4*>(p.qk + (tok0 + j) * H2 + p.H + h * kHd + c * 8);
  }
#pragma unroll
  for (int b = 0; b < kPer; ++b) {
    const int i = tid + b * kAttnThreads;
    const int c = i / cpr, pos = (i - c * cpr) * 8;
    kv[kPer + b] = u32x4{0u, 0u, 0u, 0u};
    if (pos < p.Lv)
      kv[kPer + b] = *reinterpret_cast<const u32x4*>(
          p.vt + ((int64_t)n * p.H + h * kHd + c) * p.Lv + pos);
  }
#pragma unroll
  for (int b = 0; b < kPer; ++b) {
    const int i = tid + b * kAttnThreads;
    const int j = i >> 4, c = i & 15;
    *reinterpret_cast<u32x4*>(sK + j * kHd + ((c ^ (j & 7)) << 3)) = kv[b];
  }
#pragma unroll
  for (int b = 0; b < kPer; ++b) {
    const int i = tid + b * kAttnThreads;
    const int c = i / cpr, pos = (i - c * cpr) * 8;
    u32x4 w = kv[kPer + b];
    const int nv = L - pos;  // keys of this chunk inside the lattice; the rest must be zero
    if (nv < 8) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const uint32_t keep = (2 * e + 1 < nv) ? 0xffffffffu : (2 * e < nv ? 0x0000ffffu : 0u);
        w[e] &= keep;
      }
    }
    u32x2* dst = reinterpret_cast<u32x2*>(sV + c * vstride + pos);
    dst[0] = u32x2{w.x, w.y};
    dst[1] = u32x2{w.z, w.w};
  }
  const int nb = 2 * p.S - 1;
  for (int i = tid; i < nb; i += kAttnThreads) sBias[i] = p.dist[(int64_t)h * nb + i] * kLog2e;
  if (tid == 0) sBias[nb] = p.same[h] * kLog2e;
  for (int i = tid; i < Lp; i += kAttnThreads) sSlot[i] = i < L ? i / p.K : -1;
  if constexpr (ROWS) {
    __syncthreads();  // the rows read the slot and bias tables
    for (int i = tid; i < p.S * Lp; i += kAttnThreads) {
      const int sq = i / Lp, key = i - sq * Lp;
      const int sk = sSlot[key];
      float b = -__builtin_inff();
      if (sk >= 0) {
        const int d = sq - sk;
        b = sBias[d + p.S - 1] + (d == 0 ? sBias[nb] : 0.f);
      }
      sRow[i] = b;
    }
  }
  __syncthreads();

  const float zscale = kLog2e * 0.08838834764831845f;  // log2(e) / sqrt(128)
  const float same_b = sBias[nb];
  constexpr int kWaves = kAttnThreads / 64;
  for (int qc = wave; qc < nq; qc += kWaves) {
    const int q = qc * 16 + c16;
    // logits of query q (this lane's column) against keys 16t + 4g + i
    f32x4 s[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      s[t] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        const bf16x8 a = *reinterpret_cast<const bf16x8*>(
            sK + (t * 16 + c16) * kHd + (((ks * 4 + g) ^ (c16 & 7)) << 3));
        s[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, qf[ks], s[t], 0, 0, 0);
      }
      // one tile's fragments at a time (hoisting every tile's reads would take 4 NT registers)
      __builtin_amdgcn_sched_barrier(0);
    }
    if (qc + kWaves < nq) load_q(qc + kWaves);  // the next chunk's fragments, in flight
    const int sq = q < L ? q / p.K : 0;
    float mx = -__builtin_inff();
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      {
        if constexpr (ROWS) {
          const f32x4 b = *reinterpret_cast<const f32x4*>(sRow + sq * Lp + t * 16 + 4 * g);
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            s[t][i] = fmaf(s[t][i], zscale, b[i]);
            mx = fmaxf(mx, s[t][i]);
          }
        } else {
          const i32x4 sk = *reinterpret_cast<const i32x4*>(sSlot + t * 16 + 4 * g);
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            float z = -__builtin_inff();
            if (sk[i] >= 0) {
              const int d = sq - sk[i];
              z = s[t][i] * zscale + sBias[d + p.S - 1] + (d == 0 ? same_b : 0.f);
            }
            s[t][i] = z;
            mx = fmaxf(mx, z);
          }
        }
      }
    }
    mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    float sum = 0.f;
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float e = __builtin_amdgcn_exp2f(s[t][i] - mx);
          s[t][i] = e;
          sum += e;
        }
      }
    }
    sum += __shfl_xor(sum, 16, 64);
    sum += __shfl_xor(sum, 32, 64);
    const float rs = 1.0f / sum;

    // O^T = V^T P^T: the V^T rows (head dimensions) are the MFMA rows and the probabilities of
    // this lane's query the columns, so each lane ends with four consecutive dimensions of one
    // query (one 8-byte store per 16-dimension tile)
    f32x4 o[kHd / 16];
#pragma unroll
    for (int dt = 0; dt < kHd / 16; ++dt) o[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int u = 0; u < NT / 2; ++u) {
      const u32x4 pw = u32x4{pack_bf16x2(s[2 * u][0] * rs, s[2 * u][1] * rs),
                             pack_bf16x2(s[2 * u][2] * rs, s[2 * u][3] * rs),
                             pack_bf16x2(s[2 * u + 1][0] * rs, s[2 * u + 1][1] * rs),
                             pack_bf16x2(s[2 * u + 1][2] * rs, s[2 * u + 1][3] * rs)};
      const bf16x8 pb = __builtin_bit_cast(bf16x8, pw);
#pragma unroll
      for (int dt = 0; dt < kHd / 16; ++dt) {
        const uint16_t* vr = sV + (dt * 16 + c16) * vstride + u * 32 + 4 * g;
        const u32x2 lo = *reinterpret_cast<const u32x2*>(vr);
        const u32x2 hi = *reinterpret_cast<const u32x2*>(vr + 16);
        const bf16x8 va = __builtin_bit_cast(bf16x8, u32x4{lo.x, lo.y, hi.x, hi.y});
        o[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(va, pb, o[dt], 0, 0, 0);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    // lane holds query qc * 16 + c16, head dimensions dt * 16 + 4g + i
    if (q < L) {
      u32x2* dst = reinterpret_cast<u32x2*>(p.out + (tok0 + q) * p.H + h * kHd + 4 * g);
#pragma unroll
      for (int dt = 0; dt < kHd / 16; ++dt)
        dst[dt * 4] = u32x2{pack_bf16x2(o[dt][0], o[dt][1]), pack_bf16x2(o[dt][2], o[dt][3])};
    }
  }
}

template <bool ROWS, int NT>
void launch_attention_nt(const AttnArgs& at, int64_t N, size_t lds, hipStream_t stream) {
  static const hipError_t attr = hipFuncSetAttribute(
      reinterpret_cast<const void*>(lattice_attention_kernel<ROWS, NT>),
      hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
  (void)attr;
  hipLaunchKernelGGL((lattice_attention_kernel<ROWS, NT>), dim3((unsigned)(N * at.heads)),
                     dim3(kAttnThreads), lds, stream, at);
}

template <bool ROWS>
void launch_attention_rows(const AttnArgs& at, int64_t N, size_t lds, hipStream_t stream) {
  switch (at.Lp / 16) {
    case 2: launch_attention_nt<ROWS, 2>(at, N, lds, stream); break;
    case 4: launch_attention_nt<ROWS, 4>(at, N, lds, stream); break;
    case 6: launch_attention_nt<ROWS, 6>(at, N, lds, stream); break;
    case 8: launch_attention_nt<ROWS, 8>(at, N, lds, stream); break;
    case 10: launch_attention_nt<ROWS, 10>(at, N, lds, stream); break;
    case 12: launch_attention_nt<ROWS, 12>(at, N, lds, stream); break;
    case 14: launch_attention_nt<ROWS, 14>(at, N, lds, stream); break;
    default: launch_attention_nt<ROWS, 16>(at, N, lds, stream); break;
  }
}

void launch_attention(const AttnArgs& at, int64_t N, size_t lds, hipStream_t stream) {
  if (attn_bias_rows(at.Lp, at.S))
    launch_attention_rows<true>(at, N, lds, stream);
  else
    launch_attention_rows<false>(at, N, lds, stream);
}

// ---- packing ------------------------------------------------------------------------------------
// out[c][r] = in[r][c] for a bf16 matrix of R x C (both multiples of 32); 32 x 32 tiles via LDS.
__global__ __launch_bounds__(256) void transpose_bf16_kernel(const uint16_t* __restrict__ in,
                                                             uint16_t* __restrict__ out, int R,
                                                             int C) {
  __shared__ uint16_t t[32][33];
  const int c0 = blockIdx.x * 32, r0 = blockIdx.y * 32;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
  for (int y = ty; y < 32; y += 8) t[y][tx] = in[(int64_t)(r0 + y) * C + c0 + tx];
  __syncthreads();
  for (int y = ty; y < 32; y += 8) out[(int64_t)(c0 + y) * R + r0 + tx] = t[tx][y];
}

struct PackedLayout {
  size_t qkv, o, w1, w2, g_attn, g_ffn, dist, same, total;
};

inline PackedLayout packed_layout(int H, int heads, int F, int64_t S) {
  PackedLayout l;
  size_t at = 0;
  l.qkv = at; at = align_up(at + (size_t)3 * H * H * 2);
  l.o = at; at = align_up(at + (size_t)H * H * 2);
  l.w1 = at; at = align_up(at + (size_t)F * H * 2);
  l.w2 = at; at = align_up(at + (size_t)H * F * 2);
  l.g_attn = at; at = align_up(at + (size_t)H * 4);
  l.g_ffn = at; at = align_up(at + (size_t)H * 4);
  l.dist = at; at = align_up(at + (size_t)heads * (2 * S - 1) * 4);
  l.same = at; at = align_up(at + (size_t)heads * 4);
  l.total = at;
  return l;
}

inline bool sizes_ok(int H, int heads, int F, int64_t S) {
  return H >= 256 && H <= kMaxH && H % 256 == 0 && heads * kHd == H && F >= 128 && F <= kMaxF &&
         F % 128 == 0 && S >= 1 && S <= kMaxS;
}

struct WsLayout {
  size_t xn, qk, vt, ao, hs, total;
  int Lv;
};

inline WsLayout ws_layout(int64_t N, int64_t S, int K, int H, int F) {
  WsLayout w;
  const int64_t L = S * K;
  const int64_t M = N * L;
  w.Lv = (int)((L + 7) / 8 * 8);
  size_t at = 0;
  w.xn = at; at = align_up(at + (size_t)M * H * 2);
  w.qk = at; at = align_up(at + (size_t)M * 2 * H * 2);
  w.vt = at; at = align_up(at + (size_t)N * H * w.Lv * 2);
  w.ao = at; at = align_up(at + (size_t)M * H * 2);
  w.hs = at; at = align_up(at + (size_t)M * F * 2);
  w.total = at;
  return w;
}

inline bool forward_sizes_ok(int64_t N, int64_t S, int K, int H, int F) {
  if (N < 1 || K < 1 || S < 1 || S > kMaxS || S * K > kMaxL) return false;
  const int64_t M = N * S * K;
  const int64_t widest = (3 * (int64_t)H > F ? 3 * (int64_t)H : F);
  return M * widest * 4 < ((int64_t)1 << 31);
}


void launch_rmsnorm(const float* X, const float* g, uint16_t* Y, int64_t M, int H,
                    hipStream_t stream) {
  const dim3 grid((unsigned)((M + 3) / 4)), block(256);
  switch (H / 256) {
#define LILICORR_RMS(NV)                                                                   \
  case NV:                                                                                 \
    hipLaunchKernelGGL(rmsnorm_bf16_kernel<NV>, grid, block, 0, stream, X, g, Y, M);      \
    break;
    LILICORR_RMS(1) LILICORR_RMS(2) LILICORR_RMS(3) LILICORR_RMS(4) LILICORR_RMS(5)
    LILICORR_RMS(6) LILICORR_RMS(7) LILICORR_RMS(8) LILICORR_RMS(9) LILICORR_RMS(10)
    LILICORR_RMS(11) LILICORR_RMS(12) LILICORR_RMS(13) LILICORR_RMS(14) LILICORR_RMS(15)
    LILICORR_RMS(16)
#undef LILICORR_RMS
    default: break;
  }
}

}  // namespace
}  // namespace lilicorr

using namespace lilicorr;

extern "C" size_t lilicorr_scorer_packed_bytes(int H, int heads, int F, int64_t S) {
  return sizes_ok(H, heads, F, S) ? packed_layout(H, heads, F, S).total : 0;
}

extern "C" lilicorr_status lilicorr_scorer_pack(const lilicorr_scorer_layer* layer, int H,
                                                int heads, int F, int64_t S, void* packed,
                                                hipStream_t stream) {
  if (!layer || !packed) return LILICORR_ERR_INVALID_ARG;
  if (!layer->w_qkv || !layer->w_o || !layer->w_1 || !layer->w_2 || !layer->g_attn ||
      !layer->g_ffn || !layer->dist_bias || !layer->same_bias)
    return LILICORR_ERR_INVALID_ARG;
  if (!sizes_ok(H, heads, F, S)) return LILICORR_ERR_UNSUPPORTED;
  if (!aligned16(packed)) return LILICORR_ERR_ALIGNMENT;
  const PackedLayout l = packed_layout(H, heads, F, S);
  unsigned char* base = static_cast<unsigned char*>(packed);
  auto tr = [&](const uint16_t* in, size_t off, int R, int C) {
    hipLaunchKernelGGL(transpose_bf16_kernel, dim3(C / 32, R / 32), dim3(256), 0, stream, in,
                       reinterpret_cast<uint16_t*>(base + off), R, C);
  };
  tr(layer->w_qkv, l.qkv, H, 3 * H);
  tr(layer->w_o, l.o, H, H);
  tr(layer->w_1, l.w1, H, F);
  tr(layer->w_2, l.w2, F, H);
  if (hipGetLastError() != hipSuccess) return LILICORR_ERR_HIP;
  const hipMemcpyKind k = hipMemcpyDeviceToDevice;
  if (hipMemcpyAsync(base + l.g_attn, layer->g_attn, (size_t)H * 4, k, stream) != hipSuccess ||
      hipMemcpyAsync(base + l.g_ffn, layer->g_ffn, (size_t)H * 4, k, stream) != hipSuccess ||
      hipMemcpyAsync(base + l.dist, layer->dist_bias, (size_t)heads * (2 * S - 1) * 4, k,
                     stream) != hipSuccess ||
      hipMemcpyAsync(base + l.same, layer->same_bias, (size_t)heads * 4, k, stream) != hipSuccess)
    return LILICORR_ERR_HIP;
  return LILICORR_OK;
}

extern "C" size_t lilicorr_scorer_workspace_bytes(int64_t N, int64_t S, int K, int H, int F) {
  if (!sizes_ok(H, H / kHd, F, S) || !forward_sizes_ok(N, S, K, H, F)) return 0;
  return ws_layout(N, S, K, H, F).total;
}

extern "C" lilicorr_status lilicorr_scorer_forward(float* X, int64_t N, int64_t S, int K, int H,
                                                   int heads, int F, int layers,
                                                   const void* packed, void* workspace,
                                                   size_t workspace_bytes, hipStream_t stream) {
  if (!X || !packed || !workspace || layers < 0) return LILICORR_ERR_INVALID_ARG;
  if (!sizes_ok(H, heads, F, S) || !forward_sizes_ok(N, S, K, H, F))
    return LILICORR_ERR_UNSUPPORTED;
  if (!aligned16(X) || !aligned16(packed) || !aligned16(workspace)) return LILICORR_ERR_ALIGNMENT;
  const WsLayout w = ws_layout(N, S, K, H, F);
  if (workspace_bytes < w.total) return LILICORR_ERR_WORKSPACE;
  const PackedLayout pl = packed_layout(H, heads, F, S);
  const int L = (int)(S * K);
  const int64_t M = N * L;
  unsigned char* ws = static_cast<unsigned char*>(workspace);
  uint16_t* xn = reinterpret_cast<uint16_t*>(ws + w.xn);
  uint16_t* qk = reinterpret_cast<uint16_t*>(ws + w.qk);
  uint16_t* vt = reinterpret_cast<uint16_t*>(ws + w.vt);
  uint16_t* ao = reinterpret_cast<uint16_t*>(ws + w.ao);
  uint16_t* hs = reinterpret_cast<uint16_t*>(ws + w.hs);

  AttnArgs at;
  at.qk = qk; at.vt = vt; at.out = ao;
  at.S = (int)S; at.K = K; at.L = L; at.Lv = w.Lv; at.Lp = (L + 31) / 32 * 32; at.H = H;
  at.heads = heads;
  const size_t attn_lds = attn_lds_bytes(at.Lp, at.S);


  for (int li = 0; li < layers; ++li) {
    const unsigned char* lp = static_cast<const unsigned char*>(packed) + (size_t)li * pl.total;
    const uint16_t* wqkv = reinterpret_cast<const uint16_t*>(lp + pl.qkv);
    const uint16_t* wo = reinterpret_cast<const uint16_t*>(lp + pl.o);
    const uint16_t* w1 = reinterpret_cast<const uint16_t*>(lp + pl.w1);
    const uint16_t* w2 = reinterpret_cast<const uint16_t*>(lp + pl.w2);
    const float* g_attn = reinterpret_cast<const float*>(lp + pl.g_attn);
    const float* g_ffn = reinterpret_cast<const float*>(lp + pl.g_ffn);
    at.dist = reinterpret_cast<const float*>(lp + pl.dist);
    at.same = reinterpret_cast<const float*>(lp + pl.same);

    launch_rmsnorm(X, g_attn, xn, M, H, stream);
    GemmArgs g{};
    g.A = xn; g.Bt = wqkv; g.M = M; g.K = H; g.N = 3 * H; g.Y = qk; g.Vt = vt; g.H = H; g.L = L;
    g.Lv = w.Lv;
    launch_gemm<kModeQKV>(g, stream);
    launch_attention(at, N, attn_lds, stream);
    GemmArgs r{};
    r.A = ao; r.Bt = wo; r.M = M; r.K = H; r.N = H; r.X = X;
    launch_gemm<kModeResid>(r, stream);
    launch_rmsnorm(X, g_ffn, xn, M, H, stream);
    GemmArgs f{};
    f.A = xn; f.Bt = w1; f.M = M; f.K = H; f.N = F; f.Y = hs;
    launch_gemm<kModeSilu>(f, stream);
    GemmArgs d{};
    d.A = hs; d.Bt = w2; d.M = M; d.K = F; d.N = H; d.X = X;
    launch_gemm<kModeResid>(d, stream);
  }
  return launch_status();
}
