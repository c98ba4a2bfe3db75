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
constexpr int kBM = 128, kBN = 128, kBK = 64;
constexpr int kGemmThreads = 256;
constexpr int kAttnThreads = 512;
constexpr int kMaxL = 256;
constexpr int kMaxH = 4096;
constexpr int kMaxF = 16384;
constexpr int64_t kMaxS = 256;
constexpr size_t kAlign = 256;

inline size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

__device__ __forceinline__ uint32_t bf16_rne(float x) {
  const uint32_t u = __float_as_uint(x);
  return (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
}

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return bf16_rne(lo) | (bf16_rne(hi) << 16);
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

template <int MODE>
__global__ __launch_bounds__(kGemmThreads) void gemm_bf16_kernel(GemmArgs p) {
  __shared__ __attribute__((aligned(16))) uint16_t sA[2][kBM * kBK];
  __shared__ __attribute__((aligned(16))) uint16_t sB[2][kBN * kBK];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int ntn = p.N / kBN;
  const int64_t tm = blockIdx.x / ntn;
  const int tn = (int)(blockIdx.x - tm * ntn);
  const int64_t m0 = tm * kBM;
  const int n0 = tn * kBN;
  const uint32_t K2 = (uint32_t)p.K * 2u;
  const __amdgpu_buffer_rsrc_t ra = make_rsrc(p.A, (uint32_t)p.M * K2);
  const __amdgpu_buffer_rsrc_t rb = make_rsrc(p.Bt, (uint32_t)p.N * K2);

  // staging: each thread moves chunks tid + 256 j (j = 0..3) of both 128 x 64 tiles; chunk c is
  // row c / 8, 16-byte column c % 8, stored at column (c % 8) ^ (row % 8)
  uint32_t offA[4], offB[4];
  int lds[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int c = tid + j * kGemmThreads;
    const int row = c >> 3, kc = c & 7;
    offA[j] = (uint32_t)(m0 + row) * K2 + (uint32_t)kc * 16u;
    offB[j] = (uint32_t)(n0 + row) * K2 + (uint32_t)kc * 16u;
    lds[j] = row * kBK + ((kc ^ (row & 7)) << 3);
  }
  u32x4 ga[4], gb[4];
  auto gload = [&](int k0) {
    const uint32_t kb = (uint32_t)k0 * 2u;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      ga[j] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(ra, offA[j] + kb, 0, 0));
      gb[j] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rb, offB[j] + kb, 0, 0));
    }
  };
  auto lstore = [&](int buf) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      *reinterpret_cast<u32x4*>(&sA[buf][lds[j]]) = ga[j];
      *reinterpret_cast<u32x4*>(&sB[buf][lds[j]]) = gb[j];
    }
  };

  // fragment reads: row (lane & 15) of each 16-row block, k chunk ks * 4 + lane / 16
  int rowA[4], rowB[4], sw[2];
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    rowA[t] = (wm * 64 + t * 16 + (lane & 15)) * kBK;
    rowB[t] = (wn * 64 + t * 16 + (lane & 15)) * kBK;
  }
#pragma unroll
  for (int ks = 0; ks < 2; ++ks) sw[ks] = ((ks * 4 + (lane >> 4)) ^ (lane & 7)) << 3;

  f32x4 acc[4][4];
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int b = 0; b < 4; ++b) acc[a][b] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int nk = p.K / kBK;
  gload(0);
  lstore(0);
  __syncthreads();
  for (int s = 0; s < nk; ++s) {
    const int cur = s & 1;
    if (s + 1 < nk) gload((s + 1) * kBK);
    const uint16_t* as = sA[cur];
    const uint16_t* bs = sB[cur];
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      bf16x8 a[4], b[4];
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        a[t] = *reinterpret_cast<const bf16x8*>(as + rowA[t] + sw[ks]);
        b[t] = *reinterpret_cast<const bf16x8*>(bs + rowB[t] + sw[ks]);
      }
#pragma unroll
      for (int mt = 0; mt < 4; ++mt)
#pragma unroll
        for (int nt = 0; nt < 4; ++nt)
          acc[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[mt], b[nt], acc[mt][nt], 0, 0, 0);
    }
    if (s + 1 < nk) lstore(cur ^ 1);
    __syncthreads();
  }

  // epilogue: lane holds rows 4 * (lane / 16) + j of each 16-row block, column lane % 16
  const int64_t rbase = m0 + wm * 64 + 4 * (lane >> 4);
  const int cbase = n0 + wn * 64 + (lane & 15);
#pragma unroll
  for (int mt = 0; mt < 4; ++mt)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int64_t row = rbase + mt * 16 + j;
      if (row >= p.M) continue;
#pragma unroll
      for (int nt = 0; nt < 4; ++nt) {
        const int col = cbase + nt * 16;
        const float v = acc[mt][nt][j];
        if constexpr (MODE == kModeResid) {
          float* x = p.X + row * p.N + col;
          *x = *x + v;
        } else if constexpr (MODE == kModeSilu) {
          p.Y[row * p.N + col] = (uint16_t)bf16_rne(v / (1.0f + __expf(-v)));
        } else {
          if (n0 < 2 * p.H) {
            p.Y[row * (2 * p.H) + col] = (uint16_t)bf16_rne(v);
          } else {
            const int64_t rq = row / p.L;
            const int64_t l = row - rq * p.L;
            p.Vt[(rq * p.H + (col - 2 * p.H)) * p.Lv + l] = (uint16_t)bf16_rne(v);
          }
        }
      }
    }
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

inline size_t attn_lds_bytes(int Lp, int S) {
  return (size_t)Lp * kHd * 2 + (size_t)kHd * (Lp + 4) * 2 + (size_t)((2 * S + 3) & ~3) * 4 +
         (size_t)Lp * 4;
}

__global__ __launch_bounds__(kAttnThreads) void lattice_attention_kernel(AttnArgs p) {
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  const int n = blockIdx.x / p.heads, h = blockIdx.x - n * p.heads;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int Lp = p.Lp, L = p.L, vstride = Lp + 4;
  uint16_t* sK = reinterpret_cast<uint16_t*>(smem);        // [Lp][128], chunk c of key j at c ^ (j % 8)
  uint16_t* sV = sK + Lp * kHd;                              // [128][Lp + 4]
  float* sBias = reinterpret_cast<float*>(sV + kHd * vstride);  // [2S - 1] dist, [2S - 1] same (log2 units)
  int* sSlot = reinterpret_cast<int*>(sBias + ((2 * p.S + 3) & ~3));  // [Lp] key slot, -1 past L
  const int64_t tok0 = (int64_t)n * L;
  const int H2 = 2 * p.H;

  for (int i = tid; i < Lp * 16; i += kAttnThreads) {
    const int j = i >> 4, c = i & 15;
    u32x4 v = u32x4{0u, 0u, 0u, 0u};
    if (j < L)
      v = *reinterpret_cast<const u32x4*>(p.qk + (tok0 + j) * H2 + p.H + h * kHd + c * 8);
    *reinterpret_cast<u32x4*>(sK + j * kHd + ((c ^ (j & 7)) << 3)) = v;
  }
  const int cpr = Lp / 8;
  for (int i = tid; i < kHd * cpr; i += kAttnThreads) {
    const int c = i / cpr, pos = (i - c * cpr) * 8;
    u32x4 v = u32x4{0u, 0u, 0u, 0u};
    if (pos < p.Lv)
      v = *reinterpret_cast<const u32x4*>(p.vt + ((int64_t)n * p.H + h * kHd + c) * p.Lv + pos);
    if (pos + 8 > L) {  // keys past L must contribute exactly zero
#pragma unroll
      for (int e = 0; e < 8; ++e)
        if (pos + e >= L) v[e >> 1] &= (e & 1) ? 0x0000ffffu : 0xffff0000u;
    }
    u32x2* dst = reinterpret_cast<u32x2*>(sV + c * vstride + pos);
    dst[0] = u32x2{v.x, v.y};
    dst[1] = u32x2{v.z, v.w};
  }
  const int nb = 2 * p.S - 1;
  for (int i = tid; i < nb; i += kAttnThreads) sBias[i] = p.dist[(int64_t)h * nb + i] * kLog2e;
  if (tid == 0) sBias[nb] = p.same[h] * kLog2e;
  for (int i = tid; i < Lp; i += kAttnThreads) sSlot[i] = i < L ? i / p.K : -1;
  __syncthreads();

  const float zscale = kLog2e * 0.08838834764831845f;  // log2(e) / sqrt(128)
  const float same_b = sBias[nb];
  const int nq = (L + 15) / 16, ntile = Lp / 16;
  const int g = lane >> 4, c16 = lane & 15;
  for (int qc = wave; qc < nq; qc += kAttnThreads / 64) {
    const int q = qc * 16 + c16;
    bf16x8 qf[4];
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      u32x4 v = u32x4{0u, 0u, 0u, 0u};
      if (q < L)
        v = *reinterpret_cast<const u32x4*>(p.qk + (tok0 + q) * H2 + h * kHd + ks * 32 + g * 8);
      qf[ks] = __builtin_bit_cast(bf16x8, v);
    }
    // logits of query q (this lane's column) against keys 16t + 4g + i
    f32x4 s[kMaxL / 16];
#pragma unroll
    for (int t = 0; t < kMaxL / 16; ++t) {
      s[t] = f32x4{0.f, 0.f, 0.f, 0.f};
      if (t < ntile) {
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
          const bf16x8 a = *reinterpret_cast<const bf16x8*>(
              sK + (t * 16 + c16) * kHd + (((ks * 4 + g) ^ (c16 & 7)) << 3));
          s[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, qf[ks], s[t], 0, 0, 0);
        }
      }
    }
    const int sq = q < L ? q / p.K : 0;
    float mx = -__builtin_inff();
#pragma unroll
    for (int t = 0; t < kMaxL / 16; ++t) {
      if (t < ntile) {
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
    mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    float sum = 0.f;
#pragma unroll
    for (int t = 0; t < kMaxL / 16; ++t) {
      if (t < ntile) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float e = exp2f(s[t][i] - mx);
          s[t][i] = e;
          sum += e;
        }
      }
    }
    sum += __shfl_xor(sum, 16, 64);
    sum += __shfl_xor(sum, 32, 64);
    const float rs = 1.0f / sum;

    f32x4 o[kHd / 16];
#pragma unroll
    for (int dt = 0; dt < kHd / 16; ++dt) o[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int u = 0; u < kMaxL / 32; ++u) {
      if (2 * u < ntile) {
        const u32x4 pw = u32x4{pack_bf16x2(s[2 * u][0] * rs, s[2 * u][1] * rs),
                               pack_bf16x2(s[2 * u][2] * rs, s[2 * u][3] * rs),
                               pack_bf16x2(s[2 * u + 1][0] * rs, s[2 * u + 1][1] * rs),
                               pack_bf16x2(s[2 * u + 1][2] * rs, s[2 * u + 1][3] * rs)};
        const bf16x8 pa = __builtin_bit_cast(bf16x8, pw);
#pragma unroll
        for (int dt = 0; dt < kHd / 16; ++dt) {
          const uint16_t* vr = sV + (dt * 16 + c16) * vstride + u * 32 + 4 * g;
          const u32x2 lo = *reinterpret_cast<const u32x2*>(vr);
          const u32x2 hi = *reinterpret_cast<const u32x2*>(vr + 16);
          const bf16x8 vb = __builtin_bit_cast(bf16x8, u32x4{lo.x, lo.y, hi.x, hi.y});
          o[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(pa, vb, o[dt], 0, 0, 0);
        }
      }
    }
    // lane holds queries qc * 16 + 4g + i, head dimension dt * 16 + c16
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int qq = qc * 16 + 4 * g + i;
      if (qq >= L) continue;
      uint16_t* dst = p.out + (tok0 + qq) * p.H + h * kHd + c16;
#pragma unroll
      for (int dt = 0; dt < kHd / 16; ++dt) dst[dt * 16] = (uint16_t)bf16_rne(o[dt][i]);
    }
  }
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

template <int MODE>
void launch_gemm(const GemmArgs& a, hipStream_t stream) {
  const int64_t tiles = (a.M + kBM - 1) / kBM * (a.N / kBN);
  hipLaunchKernelGGL(gemm_bf16_kernel<MODE>, dim3((unsigned)tiles), dim3(kGemmThreads), 0, stream,
                     a);
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
  static const hipError_t attr = hipFuncSetAttribute(
      reinterpret_cast<const void*>(lattice_attention_kernel),
      hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
  (void)attr;

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
    hipLaunchKernelGGL(lattice_attention_kernel, dim3((unsigned)(N * heads)), dim3(kAttnThreads),
                       attn_lds, stream, at);
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
