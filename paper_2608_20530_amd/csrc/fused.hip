// Steps 2-4 of the path in one kernel: candidate vectors (the in/out heads' stand-in u = E[id] W,
// Sec. 3.2), batched pair scores sigma * cos (Eq. pair, one matrix per adjacent slot pair,
// Sec. 3.5) and the greedy walk with its local log-likelihoods (Sec. 3.5, Eq. localar). The
// paper's serving path runs matching and selection as one replay; here the in/out vectors never
// leave the compute unit that made them.
//
// A workgroup owns up to P = 64 / K consecutive slot pairs (t, t+1) of one request:
//  1. it gathers the embedding rows of slots t0 .. t0+P once into one bf16 LDS tile: the out side
//     (slots t0 .. t0+P-1) reads its 64 rows from the tile's start and the in side
//     (slots t0+1 .. t0+P) from K rows further on, so the P-1 slots both sides share are
//     gathered once;
//  2. half of its waves project the out rows onto W_out and half the in rows onto W_in on the bf16
//     matrix cores (exact three-term weight split), each wave owning four 16-column blocks;
//  3. the raw projections u (fp32) replace the tile in LDS, with their squared norms;
//  4. every pair's K x K block is contracted on the fp32 matrix cores from LDS and scaled:
//     S = sigma * <u_o, u_i> / (||u_o|| ||u_i||) (a zero vector scores 0);
//  5. every row (slot t+1, previous choice p) of the walk's transition table is resolved from S:
//     argmax (lowest index on ties) and -log sum exp(z - max z), and written to the workspace;
//  6. the workgroup takes a ticket; the last one of its request to finish stages the request's
//     table in LDS, follows it slot by slot and writes draft, choice and logq.
// The anchor pair (when given) has a workgroup of its own: in rows of slot 0 against anchor_out.
// The exact max-path variant (decode-rule appendix) replaces steps 5-6: every workgroup writes its
// score blocks to the workspace and the request's last workgroup runs the dynamic program over
// all of them (viterbi_block), as the paper serves both decode rules as one fused kernel each.
// The certified greedy variant flags, in step 5, every row whose fp32 winner is within a margin
// of another candidate and records the contenders; in step 6 the last workgroup decides each
// flagged row it meets on the path again in double precision (certify.hpp).
#include <hip/hip_runtime.h>
#include <atomic>
#include <mutex>
#include <type_traits>
#include <math.h>
#include <stdint.h>

#include "certify.hpp"
#include "common.hpp"
#include "handover.hpp"
#include "lilicorr.h"
#include "projection.hpp"
#include "viterbi.hpp"

namespace lilicorr {
namespace {

// Candidate rows per side per workgroup (SR): 64, or 32 / 16 when a batch is too small to give
// every compute unit a workgroup at 64 (a workgroup then holds fewer slot pairs, P = SR / K).
constexpr int kFillWorkgroups = 256;
constexpr int kFusedMaxD = 256;              // the fp32 projections of both sides fit in LDS

struct FusedPlan {
  int sr;            // candidate rows per side per workgroup (64, 32 or 16; K <= sr)
  int P;             // slot pairs per workgroup
  int groups;        // pair groups per request
  int wg;            // workgroups per request (pair groups + the anchor's)
  int ws;            // waves per side
  int astride;       // bf16 elements per gathered row in LDS
  int vstride;       // floats per projected row in LDS
  TailPlan tail;     // the last workgroup's part (table or scores, from the start of LDS)
  size_t x_bytes;    // shared region: gathered tile, then projections, then (last) the tail
  size_t lds_bytes;  // total dynamic LDS
};

inline FusedPlan fused_plan(int64_t B, int K, int d, bool exact, bool cert = false, int sr = 64) {
  FusedPlan p;
  p.sr = sr;
  const VecGeom g = vec_geom(d);
  p.P = sr / K;
  const int64_t pairs = B - 1;
  p.groups = pairs > 0 ? (int)((pairs + p.P - 1) / p.P) : 1;
  p.wg = p.groups;  // the anchor workgroup is added by the caller when present
  p.ws = g.waves;
  p.astride = g.dkp * 32 + 8;
  p.vstride = d + 4;
  const size_t a_bytes = (size_t)2 * sr * p.astride * 2;
  const size_t v_bytes = (size_t)2 * sr * p.vstride * 4;
  // the exact decode stages its scores when they fit in the region the tile and projections
  // already take (at least 64 KB)
  p.x_bytes = a_bytes > v_bytes ? a_bytes : v_bytes;
  p.tail = tail_plan(B, K, d, exact, cert, 2 * p.ws * kWave,
                     p.x_bytes > 64 * 1024 ? p.x_bytes : 64 * 1024);
  if (p.tail.bytes > p.x_bytes) p.x_bytes = p.tail.bytes;
  p.x_bytes = (p.x_bytes + 15) / 16 * 16;
  p.lds_bytes = p.x_bytes + (size_t)2 * p.ws * sr * 4  // per-wave partial norms
                + (size_t)2 * sr * 4                   // row squared norms
                + (size_t)2 * sr * 4                   // row token ids
                + (size_t)p.P * K * K * 4                     // this workgroup's scores
                + 16;                                         // ticket flag
  return p;
}

template <int G, bool EXACT, bool CERT, int SR>
__global__ __launch_bounds__(512) void score_walk_kernel(
    const int32_t* __restrict__ ids, const float* __restrict__ logp,
    const uint16_t* __restrict__ E, int64_t V, int d, const unsigned char* __restrict__ frags,
    int nbp, int dkp, const float* __restrict__ anchor_out, int64_t B, int K, float sigma,
    float lambda, FusedPlan plan, float* __restrict__ S, float* __restrict__ S0,
    int32_t* __restrict__ draft, int32_t* __restrict__ choice, float* __restrict__ logq,
    float* __restrict__ score, uint32_t* __restrict__ counters, void* __restrict__ exchange,
    float margin, const float* __restrict__ w32, uint64_t* __restrict__ cmask,
    int32_t* __restrict__ rescored) {
  constexpr int kSideRows = SR, kSideRm = SR / 16;
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  uint16_t* A = reinterpret_cast<uint16_t*>(smem);  // [2 SR][astride] gathered rows
  float* Vf = reinterpret_cast<float*>(smem);       // [128][vstride] projections (after A)
  // (the last workgroup's table or scores start at smem too, after the ticket)
  uint64_t* table = static_cast<uint64_t*>(exchange);   // greedy: [N][rows] table entries
  float* xs = static_cast<float*>(exchange);            // exact: [N][rows] scores
  float* ssw = reinterpret_cast<float*>(smem + plan.x_bytes);  // [2][ws][64]
  float* nrm = ssw + 2 * plan.ws * kSideRows;                   // [128]
  int32_t* rid = reinterpret_cast<int32_t*>(nrm + 2 * kSideRows);  // [128]
  float* sbuf = reinterpret_cast<float*>(rid + 2 * kSideRows);     // [P][K][K]
  int* flag = reinterpret_cast<int*>(sbuf + plan.P * K * K);

  const int tid = threadIdx.x;
  const int nthreads = blockDim.x;
  const int nwaves = nthreads / kWave;
  const int lane = lane_id();
  const int wave = tid / kWave;
  const int64_t n = blockIdx.x / plan.wg;
  const int g = (int)(blockIdx.x % plan.wg);
  const bool anchor_wg = anchor_out != nullptr && g == plan.groups;
  const int t0 = anchor_wg ? 0 : g * plan.P;
  const int npair = anchor_wg ? 0 : (int)((B - 1 - t0) < plan.P ? (B - 1 - t0) : plan.P);
  const int n_out = npair * K;                 // out rows: slots t0 .. t0+npair-1
  const int n_in = anchor_wg ? K : npair * K;  // in rows: slots t0+1 .. (slot 0 for the anchor)
  const int dpad = dkp * 32;
  const bool use_lp = lambda != 0.f;
  const float* lpn = logp + n * B * K;

  // ---- 1. gather ------------------------------------------------------------------------------
  // wave w: local side w / ws (0: out rows on W_out, packed side 1; 1: in rows on W_in, side 0)
  const int lside = wave / plan.ws, cg = wave % plan.ws;
  const int side_rows = lside == 0 ? n_out : n_in;
  const size_t slice = (size_t)nbp * 1024;
  const unsigned char* wf = frags + (size_t)(lside == 0 ? 1 : 0) * dkp * 3 * slice +
                            (size_t)cg * kNbPerWave * 1024 + lane * 16;
  BFrag<kNbPerWave> b0;
  if (side_rows > 0) load_bfrag<kNbPerWave>(b0, wf, slice, 0);  // in flight during the gather
  // tile row r holds candidate r % K of slot s0 + r / K; the out side reads tile rows
  // [0, 64), the in side tile rows [K, K + 64). Rows outside the workgroup's slots are zero (the
  // anchor workgroup has only in rows, of slot 0: s0 = -1).
  const int tile_rows = kSideRows + K;
  const int s0 = anchor_wg ? -1 : t0;
  const int s_lo = anchor_wg ? 0 : t0, s_hi = anchor_wg ? 0 : t0 + npair;
  for (int r = tid; r < tile_rows; r += nthreads) {
    const int slot = s0 + r / K;
    int32_t id = -1;
    if (slot >= s_lo && slot <= s_hi) {
      id = ids[(n * B + slot) * K + r % K];
      if (id < 0 || id >= V) id = -1;  // outside the table: a zero row
    }
    rid[r] = id;
  }
  __syncthreads();
  gather_rows(A, plan.astride, tile_rows, rid, E, d, dpad, tid, nthreads);
  __syncthreads();

  // ---- 2. projection --------------------------------------------------------------------------
  f32x4 acc[kSideRm][kNbPerWave];
  if (side_rows > 0) {
    project_tile<kSideRm, kNbPerWave>(acc, b0, A + lside * K * plan.astride, plan.astride, wf,
                                      slice, dkp, lane);
    row_sumsq<kSideRm, kNbPerWave>(acc, ssw + (lside * plan.ws + cg) * kSideRows, lane);
  }
  __syncthreads();  // every wave is done reading the gathered tile

  // ---- 3. projections and squared norms into LDS -------------------------------------------
  for (int r = tid; r < 2 * kSideRows; r += nthreads) {
    const int rs = r / kSideRows, lr = r % kSideRows;
    float t = 0.f;
    if (lr < (rs == 0 ? n_out : n_in))
      for (int c = 0; c < plan.ws; ++c) t += ssw[(rs * plan.ws + c) * kSideRows + lr];
    nrm[r] = t;
  }
  if (side_rows > 0) {
    const int col0 = cg * kNbPerWave * 16 + (lane & 15);
#pragma unroll
    for (int mb = 0; mb < kSideRm; ++mb)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = lside * kSideRows + mb * 16 + (lane >> 4) * 4 + i;
#pragma unroll
        for (int nb = 0; nb < kNbPerWave; ++nb)
          if (col0 + nb * 16 < d) Vf[row * plan.vstride + col0 + nb * 16] = acc[mb][nb][i];
      }
  }
  __syncthreads();

  // ---- 4. scores --------------------------------------------------------------------------------
  const int r16 = lane & 15, q = lane >> 4;
  if (!anchor_wg) {
    const int nbk = (K + 15) / 16;
    const int ntiles = npair * nbk * nbk;
    for (int tile = wave; tile < ntiles; tile += nwaves) {
      const int p = tile / (nbk * nbk), bl = (tile / nbk) % nbk, br = tile % nbk;
      const int orow = p * K + bl * 16 + r16, irow = kSideRows + p * K + br * 16 + r16;
      const bool ov = bl * 16 + r16 < K, iv = br * 16 + r16 < K;
      const float* po = Vf + orow * plan.vstride + 4 * q;
      const float* pi = Vf + irow * plan.vstride + 4 * q;
      // MFMA step (s, e) contracts column 16 s + 4 q + e of both sides, into one of four
      // independent accumulators (one per e), so consecutive MFMAs never wait on each other
      f32x4 ce[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) ce[e] = f32x4{0.f, 0.f, 0.f, 0.f};
      // four steps per trip: their eight LDS reads are issued before the first MFMA
      // (d is a multiple of 16; a partial trip reads zeros)
      for (int s = 0; s < d; s += 64) {
        f32x4 a[4], b[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const bool in_d = s + 16 * u < d;
          a[u] = ov && in_d ? *reinterpret_cast<const f32x4*>(po + s + 16 * u) : f32x4{0.f, 0.f, 0.f, 0.f};
          b[u] = iv && in_d ? *reinterpret_cast<const f32x4*>(pi + s + 16 * u) : f32x4{0.f, 0.f, 0.f, 0.f};
        }
#pragma unroll
        for (int u = 0; u < 4; ++u)
#pragma unroll
          for (int e = 0; e < 4; ++e)
            ce[e] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[u][e], b[u][e], ce[e], 0, 0, 0);
      }
      const f32x4 c = (ce[0] + ce[1]) + (ce[2] + ce[3]);
      // lane (r16, q) holds rows 4 q + i, column r16 of the tile
      const int kk = br * 16 + r16;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int k = bl * 16 + 4 * q + i;
        if (k < K && kk < K) {
          const float den = sqrtf(nrm[p * K + k]) * sqrtf(nrm[kSideRows + p * K + kk]);
          sbuf[(p * K + k) * K + kk] = den > 0.f ? sigma * (c[i] / den) : 0.f;
        }
      }
    }
  } else {
    // anchor pair: S0[k'] = sigma * cos(anchor_out[n], in vector k' of slot 0)
    const float* a = anchor_out + n * d;
    for (int kk = tid; kk < K; kk += nthreads) {
      float dot = 0.f, na = 0.f;
      for (int j = 0; j < d; ++j) {
        const float x = a[j];
        dot = fmaf(x, Vf[(kSideRows + kk) * plan.vstride + j], dot);
        na = fmaf(x, x, na);
      }
      const float den = sqrtf(na) * sqrtf(nrm[kSideRows + kk]);
      sbuf[kk] = den > 0.f ? sigma * (dot / den) : 0.f;
    }
  }
  __syncthreads();

  // ---- 5. transition-table rows, or (exact decode) the score blocks; optional outputs ------
  if (EXACT) {
    float* xn = xs + n * plan.tail.rows;
    if (npair > 0)
      for (int i = tid; i < npair * K * K; i += nthreads)
        exchange_store(&xn[(int64_t)t0 * K * K + i], sbuf[i]);
    if (anchor_wg)
      for (int i = tid; i < K; i += nthreads) exchange_store(&xn[(B - 1) * (int64_t)K * K + i], sbuf[i]);
  } else {
    // rows of this workgroup: (slot t0+p+1, previous choice k) for p < npair, k < K; plus row 0
    // (slot 0) in the anchor workgroup, or in group 0 when there is no anchor
    const bool has_row0 = anchor_wg || (anchor_out == nullptr && g == 0);
    const int nrows = npair * K + (has_row0 ? 1 : 0);
    const int j = tid % G;
    const int ngroups = nthreads / G;
    const bool live = j < K;
    for (int base = 0; base < nrows; base += ngroups) {
      const int lr = base + tid / G;  // local row: 0 .. npair*K-1 pair rows, then row 0
      float z = 0.f;
      int64_t grow = -1;
      if (lr < nrows && live) {
        if (lr < npair * K) {
          const int p = lr / K;
          z = sbuf[lr * K + j];
          if (use_lp) z = fmaf(lambda, lpn[(t0 + p + 1) * K + j], z);
        } else {
          z = anchor_wg ? sbuf[j] : 0.f;
          if (use_lp) z = fmaf(lambda, lpn[j], z);
        }
      }
      if (lr < nrows) grow = lr < npair * K ? 1 + (int64_t)t0 * K + lr : 0;
      // contenders (certified): row 0 without an anchor needs none, its scores are lambda * logp
      // (or 0) on both sides of any comparison
      hand_over_row<G, CERT>(z, live, grow, lr < npair * K || anchor_wg, margin,
                             table + n * plan.tail.rows,
                             CERT ? cmask + n * plan.tail.rows : nullptr, j);
    }
  }
  {
    if (S && npair > 0) {
      float* dst = S + ((n * (B - 1) + t0) * K) * (int64_t)K;
      for (int i = tid; i < npair * K * K; i += nthreads) dst[i] = sbuf[i];
    }
    if (anchor_wg && S0)
      for (int i = tid; i < K; i += nthreads) S0[n * K + i] = sbuf[i];
  }

  // ---- 6. ticket; the request's last workgroup walks -----------------------------------------
  if (!take_ticket(&counters[n], (uint32_t)plan.wg, flag, tid, CERT && (S || S0))) return;
  TailArgs ta{n, B, V, K, d, sigma, lambda, E, w32, anchor_out, ids, logp, S, S0, draft,
              choice, logq, score, rescored, &counters[n], exchange, cmask, plan.tail};
  finish_request<G, EXACT, CERT>(ta, smem, tid, nthreads);
}

// certified greedy decode only: the re-scoring margin, the fp32 weights (the packed buffer's
// copy), the contender masks in the workspace, the optional re-scoring marks
struct CertArgs {
  float margin;
  const float* w32;
  uint64_t* cmask;
  int32_t* rescored;
};

template <int G, bool EXACT, bool CERT>
void launch_fused(const FusedPlan& plan, int64_t N, hipStream_t stream, const int32_t* ids,
                  const float* logp, const uint16_t* E, int64_t V, int d,
                  const unsigned char* frags, int nbp, int dkp, const float* anchor_out, int64_t B,
                  int K, float sigma, float lambda, float* S, float* S0, int32_t* draft,
                  int32_t* choice, float* logq, float* score, uint32_t* counters,
                  void* exchange, const CertArgs& ca) {
  auto go = [&](auto sr_const) {
    constexpr int SR = decltype(sr_const)::value;
    static const hipError_t attr = hipFuncSetAttribute(
        reinterpret_cast<const void*>(score_walk_kernel<G, EXACT, CERT, SR>),
        hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
    (void)attr;
    hipLaunchKernelGGL((score_walk_kernel<G, EXACT, CERT, SR>), dim3((unsigned)(N * plan.wg)),
                       dim3(2 * plan.ws * kWave), plan.lds_bytes, stream, ids, logp, E, V, d,
                       frags, nbp, dkp, anchor_out, B, K, sigma, lambda, plan, S, S0, draft,
                       choice, logq, score, counters, exchange, ca.margin, ca.w32, ca.cmask,
                       ca.rescored);
  };
  // K <= G <= SR: the instances with SR below G are never launched
  if constexpr (G <= 16)
    if (plan.sr == 16) return go(std::integral_constant<int, 16>{});
  if constexpr (G <= 32)
    if (plan.sr == 32) return go(std::integral_constant<int, 32>{});
  go(std::integral_constant<int, 64>{});
}

template <bool EXACT, bool CERT, bool CHECK_ONLY = false>
lilicorr_status score_and_decode(const int32_t* ids, const float* logp, const void* E,
                                 lilicorr_dtype e_dtype, int64_t V, int d, const void* packed_w,
                                 const float* anchor_out, int64_t N, int64_t B, int K, float sigma,
                                 float logp_weight, float margin, float* S, float* S0,
                                 int32_t* draft, int32_t* choice, float* logq, float* score,
                                 int32_t* rescored, void* workspace, size_t workspace_bytes,
                                 hipStream_t stream) {
  if (!ids || !logp || !E || !packed_w || !draft || !workspace) return LILICORR_ERR_INVALID_ARG;
  if (e_dtype != LILICORR_F32 && e_dtype != LILICORR_BF16) return LILICORR_ERR_INVALID_ARG;
  if (N < 1 || B < 1 || K < 1 || V < 1 || d < 1) return LILICORR_ERR_INVALID_ARG;
  if (!isfinite(sigma) || !isfinite(logp_weight)) return LILICORR_ERR_INVALID_ARG;
  if (CERT && !(isfinite(margin) && margin >= 0.f)) return LILICORR_ERR_INVALID_ARG;
  if (e_dtype != LILICORR_BF16) return LILICORR_ERR_UNSUPPORTED;
  if (d % 16 != 0 || d > kFusedMaxD || V >= ((int64_t)1 << 31)) return LILICORR_ERR_UNSUPPORTED;
  if (!decode_shape_ok(N, B, K, EXACT)) return LILICORR_ERR_UNSUPPORTED;
  if (!aligned16(ids) || !aligned16(logp) || !aligned16(E) || !aligned16(packed_w) ||
      !aligned16(draft) || !aligned16(workspace) || (anchor_out && !aligned16(anchor_out)) ||
      (S && !aligned16(S)) || (S0 && !aligned16(S0)) || (choice && !aligned16(choice)) ||
      (logq && !aligned16(logq)) || (score && !aligned16(score)) ||
      (rescored && !aligned16(rescored)))
    return LILICORR_ERR_ALIGNMENT;
  if (workspace_bytes < decode_workspace_bytes(N, B, K, EXACT, CERT)) return LILICORR_ERR_WORKSPACE;
  // the largest rows-per-side that still gives the chip kFillWorkgroups workgroups (or 16 rows,
  // the smallest block, when even that does not); never below K
  int sr = 64;
  while (sr > 16 && sr / 2 >= K &&
         N * (fused_plan(B, K, d, EXACT, CERT, sr).wg + (anchor_out ? 1 : 0)) < kFillWorkgroups)
    sr /= 2;
  FusedPlan plan = fused_plan(B, K, d, EXACT, CERT, sr);
  if (anchor_out) plan.wg += 1;
  if (N > 0x7fffffffll / plan.wg) return LILICORR_ERR_UNSUPPORTED;
  if (plan.lds_bytes > 160 * 1024) return LILICORR_ERR_UNSUPPORTED;
  if (CHECK_ONLY) return LILICORR_OK;
  const VecGeom g = vec_geom(d);
  unsigned char* ws = static_cast<unsigned char*>(workspace);
  uint32_t* counters = reinterpret_cast<uint32_t*>(ws);
  void* exchange = ws + counter_bytes(N);
  const uint16_t* e16 = static_cast<const uint16_t*>(E);
  const unsigned char* frags = static_cast<const unsigned char*>(packed_w);
  CertArgs ca{margin, nullptr, nullptr, rescored};
  if (CERT) {
    ca.w32 = reinterpret_cast<const float*>(frags + frag_bytes(d));
    ca.cmask = static_cast<uint64_t*>(exchange) + N * plan.tail.rows;
  }
  if (K <= 16)
    launch_fused<16, EXACT, CERT>(plan, N, stream, ids, logp, e16, V, d, frags, g.nbp, g.dkp,
                                  anchor_out, B, K, sigma, logp_weight, S, S0, draft, choice,
                                  logq, score, counters, exchange, ca);
  else if (K <= 32)
    launch_fused<32, EXACT, CERT>(plan, N, stream, ids, logp, e16, V, d, frags, g.nbp, g.dkp,
                                  anchor_out, B, K, sigma, logp_weight, S, S0, draft, choice,
                                  logq, score, counters, exchange, ca);
  else
    launch_fused<64, EXACT, CERT>(plan, N, stream, ids, logp, e16, V, d, frags, g.nbp, g.dkp,
                                  anchor_out, B, K, sigma, logp_weight, S, S0, draft, choice,
                                  logq, score, counters, exchange, ca);
  return launch_status();
}

// ---- allocation-free variant of the greedy pass -------------------------------------------------
// Its counters and table live in `scratch`, a file-scope device array (one copy per GPU, held
// until the process ends). Host code never passes the array's name to a kernel: at the first call
// on a device, with that device current, the array's device address is looked up once and kept
// per device; every later use goes through that address.
constexpr size_t kNoAllocScratchBytes = (size_t)8 << 20;
static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

constexpr int kMaxDevices = 64;
std::atomic<unsigned char*> g_scratch_ptr[kMaxDevices];
std::mutex g_scratch_mu;

// The device address of `scratch` on the current device, looked up once per device; null (and
// *err set) if the lookup fails.
unsigned char* scratch_address(lilicorr_status* err) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) {
    *err = LILICORR_ERR_HIP;
    return nullptr;
  }
  unsigned char* p = g_scratch_ptr[dev].load(std::memory_order_acquire);
  if (p) return p;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  p = g_scratch_ptr[dev].load(std::memory_order_relaxed);
  if (!p) {
    void* addr = nullptr;
    if (hipGetSymbolAddress(&addr, HIP_SYMBOL(scratch)) != hipSuccess || !addr) {
      *err = LILICORR_ERR_HIP;
      return nullptr;
    }
    p = static_cast<unsigned char*>(addr);
    g_scratch_ptr[dev].store(p, std::memory_order_release);
  }
  return p;
}

// Zeroes n 32-bit words (the ticket counters) before the pass: a kernel rather than a memset, so
// the call can be recorded into a graph.
__global__ __launch_bounds__(256) void clear_words_kernel(uint32_t* __restrict__ p, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256)
    p[i] = 0u;
}

}  // namespace
}  // namespace lilicorr

using namespace lilicorr;

extern "C" lilicorr_status lilicorr_score_walk_noalloc(
    const int32_t* ids, const float* logp, const void* E, lilicorr_dtype e_dtype, int64_t V, int d,
    const void* packed_w, const float* anchor_out, int64_t N, int64_t B, int K, float sigma,
    float logp_weight, float* S, float* S0, int32_t* draft, int32_t* choice, float* logq,
    hipStream_t stream) {
  // the limits and argument checks of lilicorr_score_walk come first (its own status codes);
  // then the scratch size
  if (!ids || !logp || !E || !packed_w || !draft) return LILICORR_ERR_INVALID_ARG;
  if (!decode_shape_ok(N, B, K, false)) return N < 1 || B < 1 || K < 1 ? LILICORR_ERR_INVALID_ARG
                                                                        : LILICORR_ERR_UNSUPPORTED;
  const size_t need = decode_workspace_bytes(N, B, K, false);
  if (need > kNoAllocScratchBytes) return LILICORR_ERR_WORKSPACE;
  lilicorr_status err = LILICORR_OK;
  unsigned char* ws = scratch_address(&err);
  if (!ws) return err;
  // validate everything before launching the clear (a rejected call launches nothing)
  const lilicorr_status pre = score_and_decode<false, false, true>(
      ids, logp, E, e_dtype, V, d, packed_w, anchor_out, N, B, K, sigma, logp_weight, 0.f, S, S0,
      draft, choice, logq, nullptr, nullptr, ws, need, stream);
  if (pre != LILICORR_OK) return pre;
  const int64_t words = (int64_t)(counter_bytes(N) / 4);
  hipLaunchKernelGGL(clear_words_kernel, dim3((unsigned)((words + 255) / 256 < 64 ? (words + 255) / 256 : 64)),
                     dim3(256), 0, stream, reinterpret_cast<uint32_t*>(ws), words);
  if (launch_status() != LILICORR_OK) return LILICORR_ERR_HIP;
  return score_and_decode<false, false>(ids, logp, E, e_dtype, V, d, packed_w, anchor_out, N, B,
                                        K, sigma, logp_weight, 0.f, S, S0, draft, choice, logq,
                                        nullptr, nullptr, ws, need, stream);
}

extern "C" size_t lilicorr_score_walk_workspace_bytes(int64_t N, int64_t B, int K) {
  return decode_shape_ok(N, B, K, false) ? decode_workspace_bytes(N, B, K, false) : 0;
}

extern "C" lilicorr_status lilicorr_score_walk(
    const int32_t* ids, const float* logp, const void* E, lilicorr_dtype e_dtype, int64_t V, int d,
    const void* packed_w, const float* anchor_out, int64_t N, int64_t B, int K, float sigma,
    float logp_weight, float* S, float* S0, int32_t* draft, int32_t* choice, float* logq,
    void* workspace, size_t workspace_bytes, hipStream_t stream) {
  return score_and_decode<false, false>(ids, logp, E, e_dtype, V, d, packed_w, anchor_out, N, B,
                                        K, sigma, logp_weight, 0.f, S, S0, draft, choice, logq,
                                        nullptr, nullptr, workspace, workspace_bytes, stream);
}

extern "C" size_t lilicorr_score_walk_certified_workspace_bytes(int64_t N, int64_t B, int K) {
  return decode_shape_ok(N, B, K, false) ? decode_workspace_bytes(N, B, K, false, true) : 0;
}

extern "C" lilicorr_status lilicorr_score_walk_certified(
    const int32_t* ids, const float* logp, const void* E, lilicorr_dtype e_dtype, int64_t V, int d,
    const void* packed_w, const float* anchor_out, int64_t N, int64_t B, int K, float sigma,
    float logp_weight, float margin, float* S, float* S0, int32_t* draft, int32_t* choice,
    float* logq, int32_t* rescored, void* workspace, size_t workspace_bytes, hipStream_t stream) {
  return score_and_decode<false, true>(ids, logp, E, e_dtype, V, d, packed_w, anchor_out, N, B, K,
                                       sigma, logp_weight, margin, S, S0, draft, choice, logq,
                                       nullptr, rescored, workspace, workspace_bytes, stream);
}

extern "C" size_t lilicorr_score_viterbi_workspace_bytes(int64_t N, int64_t B, int K) {
  return decode_shape_ok(N, B, K, true) ? decode_workspace_bytes(N, B, K, true) : 0;
}

extern "C" lilicorr_status lilicorr_score_viterbi(
    const int32_t* ids, const float* logp, const void* E, lilicorr_dtype e_dtype, int64_t V, int d,
    const void* packed_w, const float* anchor_out, int64_t N, int64_t B, int K, float sigma,
    float logp_weight, float* S, float* S0, int32_t* draft, int32_t* choice, float* logq,
    float* score, void* workspace, size_t workspace_bytes, hipStream_t stream) {
  return score_and_decode<true, false>(ids, logp, E, e_dtype, V, d, packed_w, anchor_out, N, B, K,
                                       sigma, logp_weight, 0.f, S, S0, draft, choice, logq, score,
                                       nullptr, workspace, workspace_bytes, stream);
}
