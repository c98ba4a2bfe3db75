// The end of a request in the one-pass decode kernels: every workgroup of a request hands its
// part of the decode over through the workspace, takes a ticket, and the request's last
// workgroup finishes the decode (Sec. 3.5: the walk follows the pair matrices of the whole block;
// the decode-rule appendix: the exact max-path decode over the same matrices).
//
// Workspace of a call: one 32-bit ticket counter per request (zero between calls), then the
// exchange region:
//   greedy     [N][1 + (B-1) K] transition-table entries (low word: the argmax, high word: the
//              fp32 local log-likelihood), row 0 for slot 0 and row 1 + (t-1) K + p for slot t
//              after choice p; certified also [N][rows] contender masks (bit k: candidate k);
//   exact      [N][(B-1) K K + K] pair scores, the slot pairs' K x K blocks then the anchor row.
// Everything the last workgroup reads goes out with device-coherent stores, so the hand-over
// needs no write-back of a compute unit's L2.
#pragma once

#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "certify.hpp"
#include "common.hpp"
#include "viterbi.hpp"

namespace lilicorr {

constexpr int64_t kMaxTableRows = 16384;          // greedy: the request's table is staged in LDS
constexpr int64_t kMaxExactSlots = 8192;          // exact decode: B bytes of path in LDS
constexpr int64_t kMaxExactBackPointers = 65536;  // exact decode: B * K bytes of predecessors
constexpr size_t kCounterBytes = 256;             // counters are padded to this alignment

inline bool decode_shape_ok(int64_t N, int64_t B, int K, bool exact) {
  if (N < 1 || B < 1 || K < 1 || K > 64) return false;
  if (exact) return B <= kMaxExactSlots && B * K <= kMaxExactBackPointers;
  return B <= kMaxTableRows && 1 + (B - 1) * (int64_t)K <= kMaxTableRows;
}

inline size_t counter_bytes(int64_t N) {
  return ((size_t)N * 4 + kCounterBytes - 1) / kCounterBytes * kCounterBytes;
}

inline size_t decode_workspace_bytes(int64_t N, int64_t B, int K, bool exact, bool cert = false) {
  if (exact) return counter_bytes(N) + (size_t)N * (size_t)((B - 1) * K * K + K) * 4;
  return counter_bytes(N) + (size_t)N * (size_t)(1 + (B - 1) * K) * 8 * (cert ? 2 : 1);
}

// LDS layout of the last workgroup's part, from the start of the dynamic LDS
struct TailPlan {
  int64_t rows;     // greedy: table rows 1 + (B-1) K; exact: floats per request in the exchange
  bool stage;       // exact: the request's scores are staged (transposed) in LDS
  size_t cert_off;  // certified: offset of the re-scoring scratch
  size_t bytes;     // LDS bytes the last workgroup needs
};

// stage_limit: LDS bytes the exact decode may use with its scores staged (it reads them from the
// workspace otherwise)
inline TailPlan tail_plan(int64_t B, int K, int d, bool exact, bool cert, int nthreads,
                          size_t stage_limit) {
  TailPlan p;
  p.cert_off = 0;
  if (exact) {
    p.rows = (B - 1) * K * K + K;
    const int G = K <= 16 ? 16 : (K <= 32 ? 32 : 64);
    const size_t s_bytes = (size_t)(B - 1) * K * (G + 4) * 4;  // transposed, padded to G + 4
    const size_t other = 64 * 8 + (size_t)(B * K + B);
    p.stage = other + s_bytes <= stage_limit;
    p.bytes = other + (p.stage ? s_bytes : 0);
  } else {
    p.rows = 1 + (B - 1) * K;
    p.stage = false;
    // table, then per slot: choice, logq (and the re-scoring mark when certified)
    p.bytes = (size_t)p.rows * 8 + (size_t)B * (cert ? 12 : 8);
    if (cert) {
      p.cert_off = (p.bytes + 15) / 16 * 16;
      p.bytes = p.cert_off + cert_scratch_bytes(d, nthreads);
    }
  }
  return p;
}

template <typename T>
__device__ __forceinline__ void exchange_store(T* p, T v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// One transition-table row resolved by a group of G lanes, one lane per candidate (lane j of the
// group holds z for candidate j; `live` is j < K), and handed over: argmax (lowest index on ties)
// and -log sum exp(z - max z) (resolve_row). grow is the row's index in the request's table, or
// -1 when the group has no row this round. Certified: a row whose fp32 winner is within `margin`
// of another candidate is flagged and its contenders handed over, unless `scored` is false (a
// row whose node scores carry no matching score: slot 0 without an anchor).
template <int G, bool CERT>
__device__ __forceinline__ void hand_over_row(float z, bool live, int64_t grow, bool scored,
                                              float margin, uint64_t* table_n, uint64_t* cmask_n,
                                              int j) {
  int arg;
  float lq, m;
  resolve_row<G>(z, live, arg, lq, m);
  uint32_t lo = (uint32_t)arg;
  uint64_t cont = 0;
  if (CERT) {
    const int gshift = (lane_id() / G) * G;
    const uint64_t gmask = G == 64 ? ~0ull : ((1ull << G) - 1);
    cont = (__ballot(live && z >= m - margin) >> gshift) & gmask;
    if (scored && __popcll(cont) > 1) lo |= kCertFlag;
  }
  if (j == 0 && grow >= 0) {
    exchange_store(&table_n[grow], (uint64_t)lo | ((uint64_t)__float_as_uint(lq) << 32));
    if (CERT && (lo & kCertFlag)) exchange_store(&cmask_n[grow], cont);
  }
}

// Every thread of the workgroup calls this after its exchange stores. Each wave waits for its own
// stores to complete (device-coherent stores are then visible to the whole device); one thread
// takes the ticket. With `release` (the certified rule when pair scores are written out) it also
// releases with a device-wide fence, because the last workgroup may overwrite pair scores the
// others wrote with ordinary stores. Only the request's last workgroup acquires (a device-wide
// fence in every workgroup would invalidate cached data under the workgroups still running).
// Returns true in every thread of the request's last workgroup.
__device__ __forceinline__ bool take_ticket(uint32_t* counter, uint32_t nwg, int* flag, int tid,
                                            bool release) {
  __asm__ volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  if (tid == 0) {
    if (release) __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
    const uint32_t done =
        __hip_atomic_fetch_add(counter, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    *flag = done == nwg - 1;
    if (*flag) __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
  }
  __syncthreads();
  return *flag != 0;
}

// What the request's last workgroup needs
struct TailArgs {
  int64_t n, B, V;
  int K, d;
  float sigma, lambda;
  const uint16_t* E;        // certified: bf16 embedding rows
  const float* w32;         // certified: fp32 W_in then W_out, [d][d] each
  const float* anchor_out;  // [N][d] or null
  const int32_t* ids;       // [N][B][K]
  const float* logp;        // [N][B][K]
  float* S;                 // optional outputs (certified: re-scored entries overwritten)
  float* S0;
  int32_t* draft;
  int32_t* choice;
  float* logq;
  float* score;             // exact
  int32_t* rescored;        // certified
  uint32_t* counter;        // this request's ticket counter
  void* exchange;           // the exchange region of the workspace
  const uint64_t* cmask;    // certified: contender masks [N][rows]
  TailPlan plan;
};

// The decode of request a.n by its last workgroup, from the hand-over in the workspace; leaves the
// request's counter at zero for the next call (visible to it at the kernel boundary).
template <int G, bool EXACT, bool CERT>
__device__ __forceinline__ void finish_request(const TailArgs& a, unsigned char* smem, int tid,
                                               int nthreads) {
  const int64_t n = a.n, B = a.B;
  const int K = a.K;
  const float* lpn = a.logp + n * B * K;
  if (EXACT) {
    const float* xn = static_cast<const float*>(a.exchange) + n * a.plan.rows;
    const int64_t nS = (B - 1) * (int64_t)K * K;
    double* line = reinterpret_cast<double*>(smem);     // [64] best path sums of one slot
    float* T = reinterpret_cast<float*>(line + kWave);  // [B-1][K][G+4] when staged
    uint8_t* from = reinterpret_cast<uint8_t*>(
        T + (a.plan.stage ? (B - 1) * (int64_t)K * viterbi_stride<G>() : 0));
    const float* S0n = a.anchor_out ? xn + nS : nullptr;
    int32_t* choice_n = a.choice ? a.choice + n * B : nullptr;
    float* logq_n = a.logq ? a.logq + n * B : nullptr;
    float* score_n = a.score ? a.score + n : nullptr;
    if (a.plan.stage) {
      if (B > 1) stage_transposed<G>(T, xn, B, K, tid, nthreads);
      __syncthreads();
      viterbi_block<G, true>(T, S0n, lpn, a.ids + n * B * K, B, K, a.lambda, from, from + B * K,
                             line, a.draft + n * B, choice_n, logq_n, score_n, tid, nthreads);
    } else {
      viterbi_block<G, false>(xn, S0n, lpn, a.ids + n * B * K, B, K, a.lambda, from,
                              from + B * K, line, a.draft + n * B, choice_n, logq_n, score_n, tid,
                              nthreads);
    }
    if (tid == 0) *a.counter = 0u;
    return;
  }
  const uint64_t* table = static_cast<const uint64_t*>(a.exchange) + n * a.plan.rows;
  uint64_t* tbl = reinterpret_cast<uint64_t*>(smem);  // [rows] the request's table
  for (int64_t i = tid; i < a.plan.rows; i += nthreads) tbl[i] = table[i];
  int32_t* ch = reinterpret_cast<int32_t*>(tbl + a.plan.rows);  // [B]
  float* lq_t = reinterpret_cast<float*>(ch + B);               // [B]
  int32_t* rs_t = reinterpret_cast<int32_t*>(lq_t + B);         // [B] (certified)
  __syncthreads();
  if (CERT) {
    // every thread follows the table (same entries, so the same branches); a flagged row on the
    // path is decided again by the whole workgroup
    const float* w_in = a.w32;
    const float* w_out = a.w32 + (size_t)a.d * a.d;
    const int32_t* idn = a.ids + n * B * K;
    int c = 0;
    for (int64_t t = 0; t < B; ++t) {
      const int64_t row = t == 0 ? 0 : 1 + (t - 1) * K + c;
      const uint64_t e = tbl[row];
      int arg = (int)((uint32_t)e & kArgMask);
      float lq = __uint_as_float((uint32_t)(e >> 32));
      int mark = 0;
      if ((uint32_t)e & kCertFlag) {
        float dlq;
        const int best = certify_decision(
            t == 0 ? a.anchor_out + n * a.d : nullptr, t == 0 ? -1 : idn[(t - 1) * K + c],
            idn + t * K, lpn + t * K, a.cmask[n * a.plan.rows + row], arg, a.E, a.V, a.d, w_in,
            w_out, a.sigma, a.lambda,
            t == 0 ? (a.S0 ? a.S0 + n * K : nullptr)
                   : (a.S ? a.S + ((n * (B - 1) + t - 1) * K + c) * (int64_t)K : nullptr),
            smem + a.plan.cert_off, tid, nthreads, dlq);
        mark = best == arg ? 1 : 2;
        arg = best;
        lq += dlq;
      }
      if (tid == 0) {
        ch[t] = arg;
        lq_t[t] = lq;
        rs_t[t] = mark;
      }
      c = arg;
    }
    if (tid == 0) *a.counter = 0u;
  } else if (tid == 0) {
    int c = 0;
    for (int64_t t = 0; t < B; ++t) {
      const uint64_t e = tbl[t == 0 ? 0 : 1 + (t - 1) * K + c];
      c = (int)(uint32_t)e;
      ch[t] = c;
      lq_t[t] = __uint_as_float((uint32_t)(e >> 32));
    }
    *a.counter = 0u;
  }
  __syncthreads();
  for (int64_t t = tid; t < B; t += nthreads) {
    const int ct = ch[t];
    a.draft[n * B + t] = a.ids[(n * B + t) * K + ct];
    if (a.choice) a.choice[n * B + t] = ct;
    if (a.logq) a.logq[n * B + t] = lq_t[t];
    if (CERT && a.rescored) a.rescored[n * B + t] = rs_t[t];
  }
}

}  // namespace lilicorr
