// Step 1 of the path: vocabulary-wide log-normalisation fused with exact top-K selection
// (Sec. 3.2 candidate pool; implementation appendix, "Serving": normalisation and candidate
// extraction in one kernel).
//
// Design (gfx950), one workgroup per row segment, four waves:
//  * Three producer waves stream the logits from HBM exactly once with 16-byte non-temporal
//    buffer loads, in interleaved tiles of 64 lanes x 32 elements (4 KB of bf16); each wave
//    issues its next tile's loads before it processes the current one.
//  * Log-sum-exp: every element adds exp2(x*log2e - c) to a per-lane partial sum; c is a
//    wave-uniform integer reference (log2 units), so moving it only rescales the partial sums by
//    an exact power of two. c is set from the producer's first tile with a finite element (its
//    maximum) and raised to a tile's maximum only when that tile's sum would exceed 2^64. Both
//    depend on the producer's own data alone (not on when the threshold moves), so the sums, and
//    the log-probabilities, are the same on every run.
//  * Top-K: a wave-uniform threshold key T (published in LDS) screens every 16-byte chunk of a
//    tile. bf16 chunks are screened with packed 16-bit integer max on the raw bit patterns (five
//    instructions per 8 elements). The screen is strict (x > value of T) whenever every id in the
//    tile exceeds T's id, which keeps runs of exactly tied logits out. A chunk that passes is
//    copied whole, with its first id and a mask of its real elements, into the producer's
//    single-producer ring in LDS (one 16-byte and one 8-byte store, slots assigned by ballot +
//    mbcnt): the producer never branches per element, which keeps its vector issue, the bound of
//    this kernel, on the stream.
//  * The fourth wave is the consumer, at raised issue priority: it drains the rings, drops chunks
//    whose maximum has fallen below the current threshold, expands the rest into (value, id) keys
//    and keeps the one sorted list of the row's K best keys in registers (one key per lane,
//    insertion by DPP lane shift, or a bitonic sort + merge when many keys arrive at once); it
//    publishes the list's K-th key as the new threshold. Each producer seeds the threshold from
//    its first tile with the K-th largest lane maximum (radix select across lanes).
//  * Every value the screen derives from T (strictness, the integer bound, the exp reference) is
//    wave-uniform and kept in scalar registers, so the per-tile control flow is scalar branches.
//  * Rows split over several workgroups (small N*B) write partial results to the workspace and a
//    second kernel merges them.
//  * Every wait (a producer for ring space, the consumer for work) is bounded by a spin limit
//    passed in at launch. A wait that gives up sets a bit in the status word at the start of the
//    caller's workspace (the kernel still runs to its end, and that call's outputs are invalid);
//    lilicorr_topk_wait_status reads and clears it.
#include <hip/hip_runtime.h>
#include <atomic>
#include <climits>
#include <type_traits>
#include <math.h>
#include <stdint.h>

#include "common.hpp"
#include "lilicorr.h"

namespace lilicorr {
namespace {

constexpr float kLog2eF = 1.44269504088896340736f;  // log2(e) rounded to fp32
constexpr int kPerLane = 32;                         // elements per lane per tile
constexpr int kTopkWaves = 4;                        // wave 0 consumes, waves 1..3 produce
constexpr int kProducers = kTopkWaves - 1;
constexpr uint32_t kRing = 256;                      // staged chunks per producer ring (power of two)
constexpr int kDefaultWaitLimit = 1 << 22;           // spins before a wait gives up (the default)
constexpr size_t kStatusBytes = 256;                 // workspace header: the wait status word
constexpr uint32_t kWaitTimedOut = 1u;               // status bit: a bounded wait gave up

// Spin limit of the waits in kernels launched from now on (lilicorr_set_wait_limit).
std::atomic<int> g_wait_limit{kDefaultWaitLimit};

__device__ __forceinline__ void report_wait_timeout(uint32_t* status) {
  if (lane_id() == 0)
    __hip_atomic_fetch_or(status, kWaitTimedOut, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef short i16x2 __attribute__((ext_vector_type(2)));

struct Partial {  // one row segment's result, written to the workspace
  int cref;
  int cvalid;
  float s;
  int pad;
  // followed by K uint64 keys
};

__host__ __device__ inline size_t partial_stride(int K) { return sizeof(Partial) + (size_t)K * 8; }

template <bool BF16>
struct ElemTraits;
template <>
struct ElemTraits<true> {
  static constexpr int kEPC = 8;  // elements per 16-byte chunk
};
template <>
struct ElemTraits<false> {
  static constexpr int kEPC = 4;
};

// A staged chunk: one lane's 16 bytes of logits that may hold a candidate, with the row-relative
// id of its first element and a mask of the elements that belong to the row segment.
struct StagedChunk {
  u32x4 raw;
  uint32_t id0;
  uint32_t mask;
  uint32_t pad[2];
};

struct TopkShared {
  uint64_t T;                      // best published threshold key (atomic max)
  uint32_t tail[kProducers];       // ring write positions (producer-owned)
  uint32_t head[kProducers];       // ring read positions (consumer-owned)
  uint32_t done;                   // producers finished
  int cref[kProducers];
  int cvalid[kProducers];
  float s[kProducers];
  StagedChunk ring[kProducers][kRing];
};

__device__ __forceinline__ uint64_t atomic_load_T(TopkShared& sh) {
  return uniform64(__hip_atomic_load(&sh.T, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP));
}

__device__ __forceinline__ void publish_T(TopkShared& sh, uint64_t t) {
  if (lane_id() == 0) atomicMax((unsigned long long*)&sh.T, (unsigned long long)t);
}

__device__ __forceinline__ int ref_for(float v) { return (int)ceilf(v * kLog2eF); }

constexpr float kBig = 0x1p64f;  // a tile sum above this is recomputed with a higher reference

// sum over the tile of exp2(x*log2e - cref), as four interleaved partial sums (short addition
// chains, few live registers)
template <int NE>
__device__ __forceinline__ float tile_exp_sum(const float (&x)[NE], int cref) {
  const float c = -(float)cref;
  if (NE >= 4) {
    // the four partial sums start from the first four terms (no additions to zero)
    float q[4];
#pragma unroll
    for (int j = 0; j < NE; ++j) {
      const float e = __builtin_amdgcn_exp2f(fmaf(x[j], kLog2eF, c));
      q[j & 3] = j < 4 ? e : q[j & 3] + e;
    }
    return (q[0] + q[1]) + (q[2] + q[3]);
  }
  float q[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int j = 0; j < NE; ++j) q[j & 3] += __builtin_amdgcn_exp2f(fmaf(x[j], kLog2eF, c));
  return (q[0] + q[1]) + (q[2] + q[3]);
}

// ---- tiles ------------------------------------------------------------------------------------

// The tiles of a row segment are read through a raw buffer descriptor bounded to the segment:
// loads past its end return zeros and touch no memory, so every load is issued unconditionally
// (no branches, exact outstanding-load counting for the prefetch) and only the segment's last,
// partial tile is padded with -inf afterwards.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t segment_rsrc(const u32x4* base, int64_t nchunks) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<u32x4*>(base), (short)0,
                                           (int)(nchunks * 16), 0x00020000);
}

template <bool BF16>
__device__ __forceinline__ void load_tile(u32x4 (&raw)[kPerLane / ElemTraits<BF16>::kEPC],
                                          __amdgpu_buffer_rsrc_t rsrc, int64_t rel_chunk0) {
  constexpr int U = kPerLane / ElemTraits<BF16>::kEPC;
  const int lane = lane_id();
  // one lane offset; the chunk-block steps (1 KB apart) go into the instruction's offset field.
  // Cache policy 3 (sc0 nt): streaming data, read once (measured fastest for this pass).
  const uint32_t base = (uint32_t)(rel_chunk0 + lane) * 16u;
#pragma unroll
  for (int u = 0; u < U; ++u)
    raw[u] = __builtin_bit_cast(
        u32x4, __builtin_amdgcn_raw_buffer_load_b128(rsrc, base + (uint32_t)u * 1024u, 0, 3));
}

template <bool BF16>
__device__ __forceinline__ void pad_tile(u32x4 (&raw)[kPerLane / ElemTraits<BF16>::kEPC],
                                         int64_t rel_chunk0, int64_t nchunks) {
  constexpr int U = kPerLane / ElemTraits<BF16>::kEPC;
  const u32x4 pad = BF16 ? u32x4{0xFF80FF80u, 0xFF80FF80u, 0xFF80FF80u, 0xFF80FF80u}
                         : u32x4{0xFF800000u, 0xFF800000u, 0xFF800000u, 0xFF800000u};
  const int lane = lane_id();
#pragma unroll
  for (int u = 0; u < U; ++u)
    if (rel_chunk0 + (int64_t)u * kWave + lane >= nchunks) raw[u] = pad;
}

template <bool BF16>
__device__ __forceinline__ void unpack_tile(const u32x4 (&raw)[kPerLane / ElemTraits<BF16>::kEPC],
                                            float (&x)[kPerLane]) {
  constexpr int U = kPerLane / ElemTraits<BF16>::kEPC;
#pragma unroll
  for (int u = 0; u < U; ++u) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      uint32_t d = raw[u][q];
      if (BF16) {
        x[u * 8 + 2 * q] = __uint_as_float(d << 16);
        x[u * 8 + 2 * q + 1] = __uint_as_float(d & 0xffff0000u);
      } else {
        x[u * 4 + q] = __uint_as_float(d);
      }
    }
  }
}

// Largest bf16 value of a 16-byte chunk (8 elements), as the signed 16-bit integer of its bit
// pattern: for positive values the integer order is the value order, and every negative pattern
// (including the -inf padding) sorts below every positive one. Packed 16-bit max over the chunk.
__device__ __forceinline__ int bf16_chunk_max(const u32x4& r) {
  // (each dword is copied to a scalar before the bit cast: a bit cast applied directly to a
  // vector element subscript has been seen to read element 0)
  const uint32_t w0 = r[0], w1 = r[1], w2 = r[2], w3 = r[3];
  const i16x2 m = __builtin_elementwise_max(
      __builtin_elementwise_max(__builtin_bit_cast(i16x2, w0), __builtin_bit_cast(i16x2, w1)),
      __builtin_elementwise_max(__builtin_bit_cast(i16x2, w2), __builtin_bit_cast(i16x2, w3)));
  return m[0] > m[1] ? (int)m[0] : (int)m[1];
}

// Element e of a 16-byte chunk as fp32.
template <bool BF16>
__device__ __forceinline__ float chunk_elem(const u32x4& r, int e) {
  if (BF16) {
    const uint32_t d = r[e >> 1];
    return __uint_as_float((e & 1) ? (d & 0xffff0000u) : (d << 16));
  }
  const uint32_t d = r[e];
  return __uint_as_float(d);
}

// ---- producer ---------------------------------------------------------------------------------

struct Producer {
  int p;            // producer index
  uint64_t seedT;   // (u) this producer's seed threshold
  uint32_t tail;    // (u) ring write position
  uint32_t head;    // (u) last ring read position seen
  int cref;         // (u) log2-units reference of the exp sums
  int cvalid;       // (u) cref is set
  float s;          // per-lane partial sum of exp2(x*log2e - cref)
  int limit;        // (u) spins before a wait for ring space gives up
  uint32_t* status; // wait status word (workspace header)
};


// Copy the chunks of the lanes with `live` set into this producer's ring (one 16-byte and one
// 8-byte LDS store per lane), waiting for ring space if the consumer is behind.
__device__ __forceinline__ void stage_chunks(Producer& pr, TopkShared& sh, const u32x4& r,
                                             uint32_t id0, uint32_t mask, bool live, uint64_t m) {
  const uint32_t n = (uint32_t)__popcll(m);
  if (pr.tail + n - pr.head > kRing) {
    // make everything written so far visible to the consumer before waiting for it
    if (lane_id() == 0)
      __hip_atomic_store(&sh.tail[pr.p], pr.tail, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
    for (int spin = 0; spin < pr.limit; ++spin) {
      pr.head = uniform32(__hip_atomic_load(&sh.head[pr.p], __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP));
      if (pr.tail + n - pr.head <= kRing) break;
      __builtin_amdgcn_s_sleep(1);
    }
    // gave up: the chunks below overwrite slots the consumer has not read (memory-safe, as the
    // ring index is masked); the call's outputs are invalid and the status word says so
    if (pr.tail + n - pr.head > kRing) report_wait_timeout(pr.status);
  }
  if (live) {
    const uint32_t off = __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
    StagedChunk& e = sh.ring[pr.p][(pr.tail + off) & (kRing - 1)];
    e.raw = r;
    *reinterpret_cast<uint2*>(&e.id0) = make_uint2(id0, mask);
  }
  pr.tail += n;
}

__device__ __forceinline__ void publish_tail(Producer& pr, TopkShared& sh) {
  if (lane_id() == 0)
    __hip_atomic_store(&sh.tail[pr.p], pr.tail, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
}

// The K-th largest lane maximum of a tile bounds the row's K-th largest element from below:
// radix select over the 32-bit order keys of the lane maxima (one compare + ballot per bit).
__device__ __forceinline__ uint64_t seed_threshold(float lane_max, int K) {
  const uint32_t lk = order_bits(lane_max);
  uint32_t prefix = 0;
#pragma unroll
  for (int b = 31; b >= 0; --b) {
    const uint32_t cand = prefix | (1u << b);
    if (__popcll(__ballot(lk >= cand)) >= K) prefix = cand;
  }
  return (uint64_t)prefix << 32;  // value = the K-th lane maximum, lowest possible id part
}

// A screen "x > Tv" is exact (no element with key > T is missed) when every element of the tile
// has a larger id than T's: then an element equal to Tv ranks below T. Otherwise "x >= Tv".
__device__ __forceinline__ bool strict_ok(uint64_t T, uint32_t tile_min_id) {
  return T != 0 && key_id(T) < tile_min_id;
}

// The producer's current threshold: the consumer's published key or this producer's own seed.
__device__ __forceinline__ uint64_t producer_T(const Producer& pr, TopkShared& sh) {
  const uint64_t T = atomic_load_T(sh);
  return uniform64(pr.seedT > T ? pr.seedT : T);
}

// Seed this producer's threshold from its first tile (lane maxima of the tile).
__device__ __forceinline__ uint64_t seed_from(Producer& pr, TopkShared& sh, uint64_t T,
                                              float lane_max, int K) {
  const uint64_t seedT = uniform64(seed_threshold(lane_max, K));
  if (key_value(seedT) > -__builtin_inff() && seedT > T) {
    // a bound for the whole row: the K lanes behind it hold K distinct elements at or above it
    pr.seedT = seedT;
    publish_T(sh, seedT);
    return seedT;
  }
  return T;
}

// Exp sums of NE elements per lane. The reference is the maximum of the producer's first tile
// with a finite element; an element far above it shows up as a tile sum beyond kBig (or inf), and
// the tile is then summed again with the reference at the tile maximum.
template <int NE>
__device__ __forceinline__ void exp_accumulate(Producer& pr, const float (&x)[NE]) {
  float lane_max = -__builtin_inff();
  bool have_max = false;
  if (!pr.cvalid) {
#pragma unroll
    for (int j = 0; j < NE; ++j) lane_max = fmaxf(lane_max, x[j]);
    have_max = true;
    const float m = wave_max_dpp(lane_max);
    if (m > -__builtin_inff()) {
      pr.cref = (int)uniform32((uint32_t)ref_for(m));
      pr.cvalid = 1;
    }
  }
  if (pr.cvalid) {
    float sum = tile_exp_sum(x, pr.cref);
    if (__ballot(!(sum <= kBig))) {
      if (!have_max) {
#pragma unroll
        for (int j = 0; j < NE; ++j) lane_max = fmaxf(lane_max, x[j]);
      }
      const int need = (int)uniform32((uint32_t)ref_for(wave_max_dpp(lane_max)));
      if (need > pr.cref) {
        pr.s = ldexpf(pr.s, pr.cref - need);
        pr.cref = need;
      }
      sum = tile_exp_sum(x, pr.cref);
    }
    pr.s += sum;
  }
}

// One full tile of U chunks per lane (chunk u of lane l holds elements tile_min_id + (u*64 + l)*EPC
// onwards). Chunks whose maximum reaches the threshold value (exceeds it when the screen is strict)
// are staged for the consumer, which tests their elements' full keys; then the exp sums.
template <bool BF16>
__device__ __forceinline__ void produce_tile(Producer& pr, TopkShared& sh,
                                             const u32x4 (&raw)[kPerLane / ElemTraits<BF16>::kEPC],
                                             uint32_t tile_min_id, uint32_t body_end_id, int K,
                                             bool first) {
  constexpr int EPC = ElemTraits<BF16>::kEPC;
  constexpr int U = kPerLane / EPC;
  const int lane = lane_id();
  float x[kPerLane];
  unpack_tile<BF16>(raw, x);
  uint64_t T = producer_T(pr, sh);
  if (first) {
    float lane_max = -__builtin_inff();
#pragma unroll
    for (int j = 0; j < kPerLane; ++j) lane_max = fmaxf(lane_max, x[j]);
    T = seed_from(pr, sh, T, lane_max, K);
  }
  T = uniform64(T);
  const float tv = key_value(T);
  // strict screen: x > value(T) (see strict_ok); on the integer bf16 patterns that is >= tb + 1.
  // Everything here derives from the wave-uniform key T, so the branches are scalar.
  const bool strict = strict_ok(T, tile_min_id);
  const uint32_t thi = (uint32_t)(T >> 32);  // order bits of the threshold value
  uint64_t mk[U];
  if (BF16 && !first && thi > 0x80000000u) {
    // positive threshold: its bf16 pattern is the high half of the fp32 bits (logits are bf16)
    const int tbe = (int)(((thi & 0x7fffffffu) >> 16) + (strict ? 1u : 0u));
    // tile maximum first (one compare); the chunks are tested only when some lane passes
    i16x2 cm2[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const uint32_t w0 = raw[u][0], w1 = raw[u][1], w2 = raw[u][2], w3 = raw[u][3];
      cm2[u] = __builtin_elementwise_max(
          __builtin_elementwise_max(__builtin_bit_cast(i16x2, w0), __builtin_bit_cast(i16x2, w1)),
          __builtin_elementwise_max(__builtin_bit_cast(i16x2, w2), __builtin_bit_cast(i16x2, w3)));
    }
    i16x2 tm = cm2[0];
#pragma unroll
    for (int u = 1; u < U; ++u) tm = __builtin_elementwise_max(tm, cm2[u]);
    const int tmax = tm[0] > tm[1] ? (int)tm[0] : (int)tm[1];
    if (__ballot(tmax >= tbe)) {
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int cm = cm2[u][0] > cm2[u][1] ? (int)cm2[u][0] : (int)cm2[u][1];
        mk[u] = __ballot(cm >= tbe);
      }
    } else {
#pragma unroll
      for (int u = 0; u < U; ++u) mk[u] = 0;
    }
  } else {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      float cm = x[u * EPC];
#pragma unroll
      for (int e = 1; e < EPC; ++e) cm = fmaxf(cm, x[u * EPC + e]);
      mk[u] = strict ? __ballot(cm > tv) : __ballot(cm >= tv);
    }
  }
  uint64_t anym = 0;
#pragma unroll
  for (int u = 0; u < U; ++u) anym |= mk[u];
  if (anym) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (!mk[u]) continue;
      const uint32_t id0 = tile_min_id + (uint32_t)((u * kWave + lane) * EPC);
      // elements past the segment end (the padded last tile) are masked out
      const int nv = (int)min(max((int64_t)body_end_id - (int64_t)id0, (int64_t)0), (int64_t)EPC);
      stage_chunks(pr, sh, raw[u], id0, (1u << nv) - 1u, (mk[u] >> lane) & 1u, mk[u]);
    }
    publish_tail(pr, sh);
  }
  exp_accumulate<kPerLane>(pr, x);
}

// ---- consumer ---------------------------------------------------------------------------------

struct Consumer {
  uint64_t L;      // this lane's entry of the sorted list (lanes >= K hold 0)
  uint64_t T_own;  // (u) key of the list's K-th entry, 0 while the list is not full
};

// Merge a batch of up to 64 keys (one per lane, 0 = none) that beat T into the list.
__device__ __forceinline__ void consume_batch(Consumer& c, TopkShared& sh, uint64_t v, uint64_t T,
                                              uint64_t m, int K) {
  const int lane = lane_id();
  const uint64_t before = c.T_own;
  if (__popcll(m) > 8) {
    // many keys: bitonic sort of the batch, then a bitonic merge with the list
    const uint64_t sorted = sort_desc64_u64(v > T ? v : 0ull);
    c.L = merge_desc64(c.L, sorted);
    if (lane >= K) c.L = 0ull;
    c.T_own = uniform64(readlane64(c.L, K - 1));
  } else {
    while (m) {
      const int ln = __ffsll((long long)m) - 1;
      const uint64_t key = readlane64(v, ln);
      const int pos = __popcll(__ballot(c.L > key));
      const uint64_t up = shift_up64(c.L);
      const uint64_t nl = lane < pos ? c.L : (lane == pos ? key : up);
      c.L = lane < K ? nl : 0ull;
      c.T_own = readlane64(c.L, K - 1);
      if (c.T_own > T) T = c.T_own;
      m &= m - 1;
      m &= __ballot(v > T);
    }
  }
  if (c.T_own > before) publish_T(sh, c.T_own);
}

// Expand a batch of staged chunks (one per lane; mask 0 = none) into keys, element position by
// element position, and merge those that beat the threshold. The threshold has usually risen
// since the chunks were staged: a lane whose chunk maximum is below its value drops out first,
// and an element position is skipped when no lane's element reaches that value.
template <bool BF16>
__device__ __forceinline__ void consume_chunks(Consumer& c, TopkShared& sh, const u32x4& r,
                                               uint32_t id0, uint32_t mask, int K) {
  constexpr int EPC = ElemTraits<BF16>::kEPC;
  uint64_t T = atomic_load_T(sh);
  if (c.T_own > T) T = c.T_own;
  T = uniform64(T);
  const uint32_t thi = (uint32_t)(T >> 32);
  if (BF16 && thi > 0x80000000u) {
    const int tb = (int)((thi & 0x7fffffffu) >> 16);
    if (bf16_chunk_max(r) < tb) mask = 0u;
  }
  if (!__ballot(mask != 0u)) return;
  const float tv = key_value(T);
#pragma unroll
  for (int e = 0; e < EPC; ++e) {
    const float v = chunk_elem<BF16>(r, e);
    const bool q = ((mask >> e) & 1u) && v >= tv;
    if (!__ballot(q)) continue;
    const uint64_t key = q ? make_key(v, id0 + (uint32_t)e) : 0ull;
    const uint64_t m = __ballot(key > T);
    if (m) {
      consume_batch(c, sh, key, T, m, K);
      if (c.T_own > T) T = uniform64(c.T_own);
    }
  }
}

// Drains the rings until every producer is done and nothing is left; a run of `limit` empty polls
// gives up and reports it in the status word.
template <bool BF16>
__device__ __forceinline__ void consume_all(Consumer& c, TopkShared& sh, int K, int limit,
                                            uint32_t* status) {
  const int lane = lane_id();
  // the consumer's batches are short and on the path of every producer's threshold: it takes
  // issue priority over the producer waves it shares a SIMD with
  __builtin_amdgcn_s_setprio(3);
  uint32_t head[kProducers];
#pragma unroll
  for (int p = 0; p < kProducers; ++p) head[p] = 0;
  bool finished = false;
  for (int idle = 0; idle < limit;) {
    bool any = false;
#pragma unroll
    for (int p = 0; p < kProducers; ++p) {
      const uint32_t t = uniform32(__hip_atomic_load(&sh.tail[p], __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP));
      while (head[p] != t) {
        const uint32_t n = t - head[p] < (uint32_t)kWave ? t - head[p] : (uint32_t)kWave;
        u32x4 r = u32x4{0u, 0u, 0u, 0u};
        uint2 im = make_uint2(0u, 0u);
        if ((uint32_t)lane < n) {
          const StagedChunk& e = sh.ring[p][(head[p] + lane) & (kRing - 1)];
          r = e.raw;
          im = *reinterpret_cast<const uint2*>(&e.id0);
        }
        head[p] += n;
        // the release orders the reads above before the slots are handed back
        if (lane == 0)
          __hip_atomic_store(&sh.head[p], head[p], __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
        consume_chunks<BF16>(c, sh, r, im.x, im.y, K);
        any = true;
      }
    }
    if (any) {
      idle = 0;
      continue;
    }
    if (__hip_atomic_load(&sh.done, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP) == (uint32_t)kProducers) {
      // every producer published its final tail before counting itself done
      bool more = false;
#pragma unroll
      for (int p = 0; p < kProducers; ++p)
        more |= uniform32(__hip_atomic_load(&sh.tail[p], __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP)) != head[p];
      if (!more) {
        finished = true;
        break;
      }
      continue;
    }
    __builtin_amdgcn_s_sleep(2);
    ++idle;
  }
  if (!finished) report_wait_timeout(status);
}

// Final outputs of a row from its merged sorted key list (one key per lane, lane 0 the best) and
// its log-sum-exp: ids and log-probabilities, and when `feat` is given the five confidence
// scalars of each candidate (implementation appendix): logp, p, the gap logp_top - logp, the rank
// k / (K-1) in [0, 1] (0 when K = 1) and the top-choice indicator. Every lane calls it.
__device__ __forceinline__ void write_row(uint64_t merged, double lse, int64_t row, int K,
                                          int32_t* ids, float* logp, float* feat) {
  const int lane = lane_id();
  const double top = (double)key_value(readlane64(merged, 0)) - lse;
  if (lane < K) {
    const double lp = (double)key_value(merged) - lse;
    ids[row * K + lane] = (int32_t)key_id(merged);
    logp[row * K + lane] = (float)lp;
    if (feat) {
      float* f = feat + (row * K + lane) * 5;
      f[0] = (float)lp;
      f[1] = (float)exp(lp);
      f[2] = (float)(top - lp);
      f[3] = K > 1 ? (float)lane / (float)(K - 1) : 0.f;
      f[4] = lane == 0 ? 1.f : 0.f;
    }
  }
}

template <bool BF16>
__global__ __launch_bounds__(kTopkWaves * kWave, 4) void topk_lse_kernel(
    const void* __restrict__ logits, int64_t V, int K, int split, int32_t* __restrict__ ids,
    float* __restrict__ logp, float* __restrict__ feat, unsigned char* __restrict__ partials,
    int wait_limit, uint32_t* __restrict__ status) {
  constexpr int EPC = ElemTraits<BF16>::kEPC;
  constexpr int U = kPerLane / EPC;
  constexpr int TILE = U * kWave;  // chunks per wave tile

  __shared__ TopkShared sh;

  const int lane = lane_id();
  const int wave = (int)uniform32(threadIdx.x / kWave);
  const int64_t row = blockIdx.x / split;
  const int part = blockIdx.x % split;
  const int64_t rowbase = row * V;
  const int64_t span = (V + split - 1) / split;
  const int64_t g0 = rowbase + (int64_t)part * span;
  const int64_t g1 = rowbase + ((int64_t)(part + 1) * span < V ? (int64_t)(part + 1) * span : V);

  if (threadIdx.x == 0) {
    sh.T = 0;
    sh.done = 0;
  }
  if (threadIdx.x < kProducers) {
    sh.tail[threadIdx.x] = 0;
    sh.head[threadIdx.x] = 0;
  }
  __syncthreads();

  // body: whole 16-byte chunks inside [g0, g1); head/tail: the ragged elements around it
  int64_t c_beg = (g0 + EPC - 1) / EPC;
  int64_t c_end = g1 / EPC;
  int n_head, n_tail;
  if (g0 < g1 && c_beg < c_end) {
    n_head = (int)(c_beg * EPC - g0);
    n_tail = (int)(g1 - c_end * EPC);
  } else {
    c_beg = c_end = 0;
    n_head = (int)(g1 > g0 ? g1 - g0 : 0);
    n_tail = 0;
  }
  const int64_t ntiles = (c_end - c_beg + TILE - 1) / TILE;
  const int64_t nchunks = c_end - c_beg;
  const __amdgpu_buffer_rsrc_t rsrc = segment_rsrc(reinterpret_cast<const u32x4*>(logits) + c_beg, nchunks);

  Consumer cons;
  cons.L = 0;
  cons.T_own = 0;
  if (wave == 0) {
    consume_all<BF16>(cons, sh, K, wait_limit, status);
  } else {
    Producer pr;
    pr.p = wave - 1;
    pr.seedT = 0;
    pr.tail = 0;
    pr.head = 0;
    pr.cref = 0;
    pr.cvalid = 0;
    pr.s = 0.f;
    pr.limit = wait_limit;
    pr.status = status;
    // producer p streams tiles p, p + 3, p + 6, ... (the workgroup reads one contiguous window
    // at a time); its tiles come in increasing id order
    const uint32_t body_end_id = (uint32_t)(c_end * EPC - rowbase);
    bool first = true;
    // one tile in flight: the next tile's loads are issued (unconditionally: past the segment end
    // the bounded descriptor returns zeros without touching memory) before the current tile is
    // processed. Two register buffers alternate (the loop is unrolled by two), so a tile is
    // processed in the registers it was loaded into rather than copied out of them.
    auto step = [&](u32x4 (&cur)[U], u32x4 (&nxt)[U], int64_t t) {
      load_tile<BF16>(nxt, rsrc, (t + kProducers) * TILE);
      if ((t + 1) * TILE > nchunks) pad_tile<BF16>(cur, t * TILE, nchunks);
      const uint32_t tile_min_id = uniform32((uint32_t)((c_beg + t * TILE) * EPC - rowbase));
      produce_tile<BF16>(pr, sh, cur, tile_min_id, body_end_id, K, first);
      first = false;
    };
    u32x4 ra[U], rb[U];
    load_tile<BF16>(ra, rsrc, (int64_t)pr.p * TILE);
    for (int64_t t = pr.p; t < ntiles; t += 2 * kProducers) {
      step(ra, rb, t);
      if (t + kProducers >= ntiles) break;
      step(rb, ra, t + kProducers);
    }
    if (wave == kTopkWaves - 1 && n_head + n_tail > 0) {
      // ragged head/tail elements, one per lane, staged as one-element chunks without a screen
      float x1[1];
      int64_t g = -1;
      if (lane < n_head) g = g0 + lane;
      else if (lane < n_head + n_tail) g = c_end * EPC + (lane - n_head);
      uint32_t bits = BF16 ? 0xFF80u : 0xFF800000u;
      if (g >= 0)
        bits = BF16 ? (uint32_t)reinterpret_cast<const uint16_t*>(logits)[g]
                    : reinterpret_cast<const uint32_t*>(logits)[g];
      x1[0] = __uint_as_float(BF16 ? bits << 16 : bits);
      uint64_t T = producer_T(pr, sh);
      if (first) T = seed_from(pr, sh, T, x1[0], K);
      const bool live = g >= 0;
      const uint64_t m = __ballot(live);
      if (m) {
        const uint32_t pad = BF16 ? 0xFF80FF80u : 0xFF800000u;
        const u32x4 r = u32x4{BF16 ? (bits | 0xFF800000u) : bits, pad, pad, pad};
        stage_chunks(pr, sh, r, (uint32_t)(g - rowbase), 1u, live, m);
        publish_tail(pr, sh);
      }
      exp_accumulate<1>(pr, x1);
    }
    const float ws = wave_sum(pr.s);
    if (lane == 0) {
      sh.cref[pr.p] = pr.cref;
      sh.cvalid[pr.p] = pr.cvalid;
      sh.s[pr.p] = ws;
      __hip_atomic_store(&sh.tail[pr.p], pr.tail, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
      __hip_atomic_fetch_add(&sh.done, 1u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
    }
  }
  __syncthreads();
  if (wave != 0) return;

  int C = 0, any = 0;
  for (int i = 0; i < kProducers; ++i)
    if (sh.cvalid[i]) {
      C = any ? (sh.cref[i] > C ? sh.cref[i] : C) : sh.cref[i];
      any = 1;
    }
  float S = 0.f;
  for (int i = 0; i < kProducers; ++i)
    if (sh.cvalid[i]) S += ldexpf(sh.s[i], sh.cref[i] - C);
  const uint64_t merged = cons.L;

  if (split == 1) {
    write_row(merged, (log2((double)S) + (double)C) / (double)kLog2eF, row, K, ids, logp, feat);
  } else {
    unsigned char* q = partials + ((size_t)row * split + part) * partial_stride(K);
    Partial* hdr = reinterpret_cast<Partial*>(q);
    uint64_t* keys = reinterpret_cast<uint64_t*>(q + sizeof(Partial));
    if (lane == 0) {
      hdr->cref = C;
      hdr->cvalid = any;
      hdr->s = S;
      hdr->pad = 0;
    }
    if (lane < K) keys[lane] = merged;
  }
}

// ---- short row segments --------------------------------------------------------------------
// Rows split over many workgroups (few rows) leave each workgroup a short segment, where the
// streaming kernel's fixed costs (producer/consumer set-up, threshold seeding, ring hand-offs)
// dominate. Segments of at most kSmallSpan logits take this kernel instead and write the same
// partial record for the merge kernel. Every thread holds 32 logits (element tid + 256 j), all
// loaded before the first is used. The workgroup reduces the maximum and the exp sum relative to
// the same integer log2 reference as the streaming kernel.
// Top-K: a threshold T that at least K of the segment's elements reach, so that its K largest
// keys all do. At K <= 8 each wave finds the K-th largest of its 64 lane maxima by a bitwise
// search over their order bits (one ballot per bit) and T is the largest of the four; at larger K
// (where that leaves more than 64 candidates on random logits) T is the K-th largest of all 256
// lane maxima (every wave reads them from LDS; four ballots per bit). The elements >= T are the
// candidates: each lane counts its own, a prefix sum over the wave places them in LDS, and wave 0
// ranks them (a key's rank is the number of larger candidates; keys are distinct) and writes the
// K largest in order. When more than 64 elements reach T (exact ties at T, such as a segment that
// is all -inf), T becomes the workgroup-wide value completed over the ids of the lane maxima (the
// smallest id holding each) where more lanes than needed hold it, which bounds the candidates by
// key; more than 64 still take a sort-and-merge loop.
constexpr int kSmallThreads = 256;
constexpr int kSmallPer = 32;
constexpr int64_t kSmallSpan = (int64_t)kSmallThreads * kSmallPer;
constexpr int kSmallFill = 512;  // workgroups that run at once (two per compute unit)
constexpr int kSmallWaveK = 8;   // largest K whose first threshold is taken per wave

// Exclusive prefix sum over the wave of a per-lane count below 64, from one ballot per bit.
__device__ __forceinline__ int wave_prefix_small(int c) {
  int p = 0;
#pragma unroll
  for (int bit = 0; bit < 6; ++bit) {
    const uint64_t bal = __ballot((c >> bit) & 1);
    p += (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(bal >> 32),
                                        __builtin_amdgcn_mbcnt_lo((uint32_t)bal, 0u)) << bit;
  }
  return p;
}

// The largest t with at least `need` lanes of the wave holding v >= t.
__device__ __forceinline__ uint32_t wave_kth_bits(uint32_t v, int need) {
  uint32_t t = 0;
#pragma unroll
  for (int bit = 31; bit >= 0; --bit) {
    const uint32_t c = t | (1u << bit);
    if (__popcll(__ballot(v >= c)) >= need) t = c;
  }
  return t;
}

// The largest t such that at least `need` of the workgroup's 256 values v[] (four per lane of
// every wave, read from LDS, so every wave finds the same t) with on[] set are >= t.
__device__ __forceinline__ uint32_t block_kth_bits(const uint32_t (&v)[4], const bool (&on)[4],
                                                   int need) {
  uint32_t t = 0;
#pragma unroll
  for (int bit = 31; bit >= 0; --bit) {
    const uint32_t c = t | (1u << bit);
    int n = 0;
#pragma unroll
    for (int i = 0; i < 4; ++i) n += __popcll(__ballot(on[i] & (v[i] >= c)));
    if (n >= need) t = c;
  }
  return t;
}

template <bool BF16>
__global__ __launch_bounds__(kSmallThreads) void topk_small_kernel(
    const void* __restrict__ logits, int64_t V, int K, int split,
    unsigned char* __restrict__ partials) {
  constexpr int NW = kSmallThreads / kWave;
  __shared__ uint64_t sCand[kSmallSpan];
  __shared__ float sMax[NW], sSum[NW];
  __shared__ uint32_t sKhi[kSmallThreads], sKlo[kSmallThreads];
  __shared__ int sCount[2];
  const int tid = threadIdx.x, lane = lane_id(), wave = tid / kWave;
  const int64_t row = blockIdx.x / split;
  const int part = blockIdx.x % split;
  const int64_t span = (V + split - 1) / split;
  const int64_t lo = (int64_t)part * span;
  const int64_t hi = lo + span < V ? lo + span : V;
  const int len = (int)(hi > lo ? hi - lo : 0);
  const int64_t base = row * V + lo;
  const int rem = len - tid;  // element j of this thread lies in the segment iff 256 j < rem
  if (tid == 0) sCount[0] = sCount[1] = 0;

  // positions past the segment load the row's first element (in bounds for any segment, even an
  // empty one) and are masked afterwards, so no load waits behind another
  float x[kSmallPer];
  const int64_t rowstart = row * V;
#pragma unroll
  for (int j = 0; j < kSmallPer; ++j) {
    const int64_t g = kSmallThreads * j < rem ? base + tid + kSmallThreads * j : rowstart;
    if constexpr (BF16)
      x[j] = __uint_as_float((uint32_t)static_cast<const uint16_t*>(logits)[g] << 16);
    else
      x[j] = static_cast<const float*>(logits)[g];
  }
  float m = -__builtin_inff();
#pragma unroll
  for (int j = 0; j < kSmallPer; ++j) {
    x[j] = kSmallThreads * j < rem ? x[j] : -__builtin_inff();
    m = fmaxf(m, x[j]);
  }
  const uint32_t khi = rem > 0 ? order_bits(m) : 0u;  // the lane's largest value (0: none)
  // the threshold: at K <= 8 the largest of the waves' K-th lane maxima (about 4K candidates),
  // else the K-th largest of all 256 lane maxima (a tighter bound for a costlier search)
  const bool per_wave = K <= kSmallWaveK;
  sKhi[tid] = khi;
  const uint32_t thi = per_wave ? wave_kth_bits(khi, K) : 0u;
  const float mw = wave_max(m);
  if (lane == 0) {
    sMax[wave] = mw;
    sKlo[wave] = thi;  // the waves' thresholds (sKlo is reused for lane ids only later)
  }
  __syncthreads();
  float M = sMax[0];
  uint32_t Thi = sKlo[0];
#pragma unroll
  for (int w = 1; w < NW; ++w) {
    M = fmaxf(M, sMax[w]);
    Thi = sKlo[w] > Thi ? sKlo[w] : Thi;
  }
  uint32_t all_hi[4];
  const bool every[4] = {true, true, true, true};
#pragma unroll
  for (int i = 0; i < 4; ++i) all_hi[i] = sKhi[lane + kWave * i];
  if (!per_wave) Thi = block_kth_bits(all_hi, every, K);
  const bool valid = M > -__builtin_inff();
  const int C = valid ? ref_for(M) : 0;
  const float c = -(float)C;
  float e = 0.f;
#pragma unroll
  for (int j = 0; j < kSmallPer; ++j) e += __builtin_amdgcn_exp2f(fmaf(x[j], kLog2eF, c));
  e = wave_sum(e);
  if (lane == 0) sSum[wave] = e;

  // candidates (value, id) >= (Tv, Tlo): value > Tv, or value == Tv and id part >= Tlo (the first
  // pass takes every id: value >= Tv). The order bits of -0 and +0 are equal, as are the values;
  // Thi = 0 (fewer than K lanes holding elements, in every wave or in the workgroup, as searched)
  // makes every element a candidate; the padding (-inf) is told apart by position when Tv is
  // -inf. Predicates use non-short-circuit operators
  // so that they compile to mask arithmetic rather than branches.
  auto place = [&](auto by_id, float Tv, uint32_t Tlo, int slot) {
    const int lim = Tv == -__builtin_inff() ? rem : kSmallThreads * kSmallPer;
    auto cand = [&](int j) {
      const bool in = kSmallThreads * j < lim;
      if constexpr (decltype(by_id)::value) {
        const uint32_t idc = 0xFFFFFFFFu - (uint32_t)(lo + tid + kSmallThreads * j);
        return in & ((x[j] > Tv) | ((x[j] == Tv) & (idc >= Tlo)));
      } else {
        return in & (x[j] >= Tv);
      }
    };
    int cnt = 0;
#pragma unroll
    for (int j = 0; j < kSmallPer; ++j) cnt += cand(j) ? 1 : 0;
    int off = wave_prefix_small(cnt);
    const int wtotal = __shfl(off + cnt, kWave - 1, kWave);
    int at = 0;
    if (lane == 0) at = atomicAdd(&sCount[slot], wtotal);
    off += __shfl(at, 0, kWave);
#pragma unroll
    for (int j = 0; j < kSmallPer; ++j)
      if (cand(j)) sCand[off++] = make_key(x[j], (uint32_t)(lo + tid + kSmallThreads * j));
  };
  place(std::false_type{}, Thi ? order_value(Thi) : -__builtin_inff(), 0u, 0);
  __syncthreads();
  int total = sCount[0];
  if (total > kWave) {
    // the K-th largest of all 256 lane maxima, then, among the lanes holding exactly that value,
    // the id bits of their keys (the smallest id holding the lane maximum)
    if (per_wave) Thi = block_kth_bits(all_hi, every, K);
    int jm = 0;
#pragma unroll
    for (int j = kSmallPer - 1; j >= 0; --j) jm = x[j] == m ? j : jm;
    sKlo[tid] = 0xFFFFFFFFu - (uint32_t)(lo + tid + kSmallThreads * jm);  // every wave read sKlo[w]
    __syncthreads();
    uint32_t Tlo = 0;
    if (Thi != 0) {
      uint32_t all_lo[4];
      bool at_t[4];
      int above = 0;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        all_lo[i] = sKlo[lane + kWave * i];
        at_t[i] = all_hi[i] == Thi;
        above += __popcll(__ballot(all_hi[i] > Thi));
      }
      Tlo = block_kth_bits(all_lo, at_t, K - above);
    }
    place(std::true_type{}, Thi ? order_value(Thi) : -__builtin_inff(), Tlo, 1);
    __syncthreads();
    total = sCount[1];
  }
  if (wave != 0) return;
  float S = 0.f;
#pragma unroll
  for (int w = 0; w < NW; ++w) S += sSum[w];
  unsigned char* q = partials + ((size_t)row * split + part) * partial_stride(K);
  Partial* hdr = reinterpret_cast<Partial*>(q);
  uint64_t* keys = reinterpret_cast<uint64_t*>(q + sizeof(Partial));
  if (lane == 0) {
    hdr->cref = C;
    hdr->cvalid = valid ? 1 : 0;
    hdr->s = valid ? S : 0.f;
    hdr->pad = 0;
  }
  if (total <= kWave) {
    const uint64_t mine = lane < total ? sCand[lane] : 0ull;
    int rank = 0;
    for (int i = 0; i < total; ++i) rank += sCand[i] > mine ? 1 : 0;
    if (lane < total && rank < K) keys[rank] = mine;
    if (lane >= total && lane < K) keys[lane] = 0ull;
  } else {
    uint64_t L = 0ull;
    for (int b = 0; b < total; b += kWave) {
      const uint64_t v = b + lane < total ? sCand[b + lane] : 0ull;
      L = b == 0 ? sort_desc64_u64(v) : merge_desc64(L, sort_desc64_u64(v));
    }
    if (lane < K) keys[lane] = L;
  }
}

// One workgroup of four waves per row merges the row's `split` (<= 256) partial results: thread
// p reads partial p's (reference, exp sum) header and the workgroup reduces them. The key lists:
//  * when the row holds at most kMergeFast entries (split K), every entry is loaded at once
//    (eight per thread). Partial p* whose K-th key is the largest, T, holds K keys >= T, so the
//    row's K largest keys all reach T: only entries >= T are candidates (usually little more
//    than K; when no partial is full, T = 0 and every key is one), compacted into LDS. Wave 0
//    ranks them (a key's rank is the number of larger candidates; keys are distinct) and places
//    the K largest in order; more than 64 candidates take a sort-and-merge loop;
//  * otherwise wave w merges the lists of partials w, w + 4, ..., eight lists' loads in flight
//    at a time, and wave 0 merges the four results through LDS.
constexpr int kMergeThreads = 256;
constexpr int kMergeBatch = 8;
constexpr int kMergeFast = kMergeThreads * kMergeBatch;

__global__ __launch_bounds__(kMergeThreads) void topk_merge_kernel(
    const unsigned char* __restrict__ partials, int K, int split, int32_t* __restrict__ ids,
    float* __restrict__ logp, float* __restrict__ feat) {
  constexpr int NW = kMergeThreads / kWave;
  __shared__ int sC[NW];
  __shared__ float sS[NW];
  __shared__ uint64_t sL[NW][kWave];
  __shared__ uint64_t sCand[kMergeFast];
  __shared__ unsigned long long sT;
  __shared__ int sCount;
  const int tid = threadIdx.x, lane = lane_id(), wave = tid / kWave;
  const int64_t row = blockIdx.x;
  const size_t stride = partial_stride(K);
  const unsigned char* base = partials + (size_t)row * split * stride;
  const int E = split * K;
  const bool fast = E <= kMergeFast;
  if (tid == 0) {
    sT = 0ull;
    sCount = 0;
  }

  // reference: the largest valid one (no valid partial: reference 0, sum 0). Every load below is
  // issued unconditionally (threads past the end read partial 0 or entry 0 and discard it), so
  // none waits behind another.
  const Partial* hdr = reinterpret_cast<const Partial*>(base + (size_t)(tid < split ? tid : 0) * stride);
  int cref = hdr->cref, valid = hdr->cvalid;
  float s = hdr->s;
  if (tid >= split) valid = 0;
  // entries tid + 256 i of the row (fast path)
  uint64_t kv[kMergeBatch];
  if (fast) {
#pragma unroll
    for (int i = 0; i < kMergeBatch; ++i) {
      const int e = tid + kMergeThreads * i < E ? tid + kMergeThreads * i : 0;
      kv[i] = reinterpret_cast<const uint64_t*>(base + (size_t)(e / K) * stride +
                                                sizeof(Partial))[e % K];
    }
  }
  int c = valid ? cref : INT_MIN;
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) {
    const int o = __shfl_xor(c, m, kWave);
    c = o > c ? o : c;
  }
  if (lane == 0) sC[wave] = c;
  __syncthreads();
  int C = sC[0];
#pragma unroll
  for (int w = 1; w < NW; ++w) C = sC[w] > C ? sC[w] : C;
  if (C == INT_MIN) C = 0;
  float part = valid ? ldexpf(s, cref - C) : 0.f;
  part = wave_sum(part);
  if (lane == 0) sS[wave] = part;

  uint64_t merged = 0;
  if (fast) {
#pragma unroll
    for (int i = 0; i < kMergeBatch; ++i) {
      const int e = tid + kMergeThreads * i;
      if (e < E && e % K == K - 1) atomicMax(&sT, (unsigned long long)kv[i]);
    }
    __syncthreads();
    const uint64_t T = sT;
    int cnt = 0;
#pragma unroll
    for (int i = 0; i < kMergeBatch; ++i) {
      const bool q = tid + kMergeThreads * i < E && kv[i] != 0ull && kv[i] >= T;
      cnt += q ? 1 : 0;
    }
    int off = wave_prefix_small(cnt);
    const int wtotal = __shfl(off + cnt, kWave - 1, kWave);
    int at = 0;
    if (lane == 0) at = atomicAdd(&sCount, wtotal);
    off += __shfl(at, 0, kWave);
#pragma unroll
    for (int i = 0; i < kMergeBatch; ++i)
      if (tid + kMergeThreads * i < E && kv[i] != 0ull && kv[i] >= T) sCand[off++] = kv[i];
    __syncthreads();
    if (wave != 0) return;
    const int total = sCount;
    if (total <= kWave) {
      const uint64_t mine = lane < total ? sCand[lane] : 0ull;
      int rank = 0;
      for (int i = 0; i < total; ++i) rank += sCand[i] > mine ? 1 : 0;
      if (lane < total && rank < K) sL[0][rank] = mine;
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
      merged = lane < K ? sL[0][lane] : 0ull;
    } else {
      for (int b = 0; b < total; b += kWave) {
        const uint64_t v = b + lane < total ? sCand[b + lane] : 0ull;
        merged = b == 0 ? sort_desc64_u64(v) : merge_desc64(merged, sort_desc64_u64(v));
      }
    }
    float S = sS[0];
#pragma unroll
    for (int w = 1; w < NW; ++w) S += sS[w];
    write_row(merged, (log2((double)S) + (double)C) / (double)kLog2eF, row, K, ids, logp, feat);
    return;
  }

  bool first = true;
  for (int p0 = wave; p0 < split; p0 += kMergeBatch * NW) {
    uint64_t k[kMergeBatch];
#pragma unroll
    for (int b = 0; b < kMergeBatch; ++b) {
      const int p = p0 + b * NW;
      k[b] = reinterpret_cast<const uint64_t*>(base + (size_t)(p < split ? p : 0) * stride +
                                               sizeof(Partial))[lane < K ? lane : 0];
    }
#pragma unroll
    for (int b = 0; b < kMergeBatch; ++b) k[b] = (p0 + b * NW < split && lane < K) ? k[b] : 0ull;
#pragma unroll
    for (int b = 0; b < kMergeBatch; ++b) {
      const int p = p0 + b * NW;
      if (p < split) {
        merged = first ? k[b] : merge_desc64(merged, k[b]);
        first = false;
      }
    }
  }
  sL[wave][lane] = merged;  // an empty list (all zero keys) when the wave had no partial
  __syncthreads();
  if (wave == 0) {
    float S = sS[0];
#pragma unroll
    for (int w = 1; w < NW; ++w) {
      S += sS[w];
      merged = merge_desc64(merged, sL[w][lane]);
    }
    write_row(merged, (log2((double)S) + (double)C) / (double)kLog2eF, row, K, ids, logp, feat);
  }
}

// Number of workgroups per row: enough workgroups to fill the chip (about four per CU), but
// no segment shorter than two workgroup tiles.
int topk_split(int64_t rows, int64_t V, bool bf16) {
  const int64_t wg_tile = (int64_t)kProducers * kWave * kPerLane;
  const int64_t target = 1024;
  int64_t by_fill = (target + rows - 1) / rows;
  int64_t by_len = V / (2 * wg_tile);
  int64_t s = by_fill < by_len ? by_fill : by_len;
  if (s < by_fill) {
    // too few rows to fill the chip with streaming segments: when every row's short segments (at
    // most kSmallSpan logits) run at once, they take the short-segment kernel
    const int64_t t = (V + kSmallSpan - 1) / kSmallSpan;
    if (t > 1 && t <= 256 && rows * t <= kSmallFill) s = t;
  }
  if (s < 1) s = 1;
  if (s > 256) s = 256;
  (void)bf16;
  return (int)s;
}

bool topk_args_ok(int64_t N, int64_t B, int64_t V, int K) {
  if (N < 1 || B < 1 || V < 1 || K < 1) return false;
  if (V >= ((int64_t)1 << 31)) return false;
  if (N > ((int64_t)1 << 40) / B) return false;
  if ((N * B) > (((int64_t)1 << 62) / V)) return false;
  return true;
}

}  // namespace
}  // namespace lilicorr

using namespace lilicorr;

// workspace: the status header, then (rows split over several workgroups) the partial results
inline size_t topk_workspace_need(int64_t rows, int split, int K) {
  return kStatusBytes + (split == 1 ? 0 : (size_t)rows * split * partial_stride(K));
}

extern "C" size_t lilicorr_topk_workspace_bytes(int64_t N, int64_t B, int64_t V, int K) {
  if (!topk_args_ok(N, B, V, K) || K > 64 || K > V) return 0;
  return topk_workspace_need(N * B, topk_split(N * B, V, true), K);
}

extern "C" lilicorr_status lilicorr_topk_wait_status(const void* workspace, hipStream_t stream) {
  if (!workspace) return LILICORR_ERR_INVALID_ARG;
  if (!aligned16(workspace)) return LILICORR_ERR_ALIGNMENT;
  uint32_t word = 0;
  if (hipStreamSynchronize(stream) != hipSuccess) return LILICORR_ERR_HIP;
  if (hipMemcpy(&word, workspace, sizeof word, hipMemcpyDeviceToHost) != hipSuccess)
    return LILICORR_ERR_HIP;
  if (word == 0) return LILICORR_OK;
  const uint32_t zero = 0;
  if (hipMemcpy(const_cast<void*>(workspace), &zero, sizeof zero, hipMemcpyHostToDevice) !=
      hipSuccess)
    return LILICORR_ERR_HIP;
  return LILICORR_ERR_TIMEOUT;
}

extern "C" void lilicorr_set_wait_limit(int64_t spins) {
  g_wait_limit.store(spins < 0 ? kDefaultWaitLimit : (int)(spins < INT_MAX ? spins : INT_MAX));
}

static lilicorr_status topk_launch(const void* logits, lilicorr_dtype dtype, int64_t N, int64_t B,
                                   int64_t V, int K, int32_t* ids, float* logp, float* feat,
                                   void* workspace, size_t workspace_bytes, hipStream_t stream) {
  if (!logits || !ids || !logp) return LILICORR_ERR_INVALID_ARG;
  if (dtype != LILICORR_F32 && dtype != LILICORR_BF16) return LILICORR_ERR_INVALID_ARG;
  if (!topk_args_ok(N, B, V, K)) return LILICORR_ERR_INVALID_ARG;
  if (K > 64 || K > V) return LILICORR_ERR_UNSUPPORTED;
  if (!aligned16(logits) || !aligned16(ids) || !aligned16(logp) || (feat && !aligned16(feat)))
    return LILICORR_ERR_ALIGNMENT;
  const bool bf16 = dtype == LILICORR_BF16;
  const int64_t rows = N * B;
  const int split = topk_split(rows, V, bf16);
  const size_t need = topk_workspace_need(rows, split, K);
  if (!workspace || workspace_bytes < need) return LILICORR_ERR_WORKSPACE;
  if (!aligned16(workspace)) return LILICORR_ERR_ALIGNMENT;
  if (rows * split > 0x7fffffffll) return LILICORR_ERR_UNSUPPORTED;

  dim3 grid((unsigned)(rows * split)), block(kTopkWaves * kWave);
  uint32_t* status = static_cast<uint32_t*>(workspace);
  unsigned char* ws = static_cast<unsigned char*>(workspace) + kStatusBytes;
  const int limit = g_wait_limit.load();
  const bool small = split > 1 && (V + split - 1) / split <= kSmallSpan;
  if (small && bf16)
    hipLaunchKernelGGL(topk_small_kernel<true>, grid, dim3(kSmallThreads), 0, stream, logits, V, K,
                       split, ws);
  else if (small)
    hipLaunchKernelGGL(topk_small_kernel<false>, grid, dim3(kSmallThreads), 0, stream, logits, V,
                       K, split, ws);
  else if (bf16)
    hipLaunchKernelGGL(topk_lse_kernel<true>, grid, block, 0, stream, logits, V, K, split, ids, logp,
                       feat, ws, limit, status);
  else
    hipLaunchKernelGGL(topk_lse_kernel<false>, grid, block, 0, stream, logits, V, K, split, ids,
                       logp, feat, ws, limit, status);
  if (launch_status() != LILICORR_OK) return LILICORR_ERR_HIP;
  if (split > 1) {
    hipLaunchKernelGGL(topk_merge_kernel, dim3((unsigned)rows), dim3(kMergeThreads), 0, stream, ws, K, split,
                       ids, logp, feat);
    if (launch_status() != LILICORR_OK) return LILICORR_ERR_HIP;
  }
  return LILICORR_OK;
}

extern "C" lilicorr_status lilicorr_topk(const void* logits, lilicorr_dtype dtype, int64_t N,
                                         int64_t B, int64_t V, int K, int32_t* ids, float* logp,
                                         void* workspace, size_t workspace_bytes,
                                         hipStream_t stream) {
  return topk_launch(logits, dtype, N, B, V, K, ids, logp, nullptr, workspace, workspace_bytes,
                     stream);
}

extern "C" lilicorr_status lilicorr_topk_features(const void* logits, lilicorr_dtype dtype,
                                                  int64_t N, int64_t B, int64_t V, int K,
                                                  int32_t* ids, float* logp, float* feat,
                                                  void* workspace, size_t workspace_bytes,
                                                  hipStream_t stream) {
  if (!feat) return LILICORR_ERR_INVALID_ARG;
  return topk_launch(logits, dtype, N, B, V, K, ids, logp, feat, workspace, workspace_bytes,
                     stream);
}
