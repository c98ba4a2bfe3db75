// Step 1 of the path: vocabulary-wide log-normalisation fused with exact top-K selection
// (Sec. 3.2 candidate pool; implementation appendix, "Serving": normalisation and candidate
// extraction in one kernel).
//
// Design (gfx950), one workgroup per row segment, four waves:
//  * Three producer waves stream the logits from HBM exactly once with 16-byte non-temporal
//    buffer loads, in interleaved tiles of 64 lanes x 32 elements (4 KB of bf16), two tiles in
//    flight per wave.
//  * Log-sum-exp: every element adds exp2(x*log2e - c) to a per-lane partial sum; c is a
//    wave-uniform integer reference (log2 units), so moving it only rescales the partial sums by
//    an exact power of two. c follows the top-K threshold value (a logit of the row, so the
//    maximum's term stays at or above 2^-1) and is raised to the tile maximum in the rare case
//    a tile sum exceeds 2^64.
//  * Top-K: a wave-uniform threshold key T (published in LDS) screens each tile. bf16 tiles are
//    screened with packed 16-bit integer max on the raw bit patterns, so a tile with no candidate
//    costs about half an instruction per element. The screen is strict (x > value of T) whenever
//    every id in the tile exceeds T's id, which keeps runs of exactly tied logits out. Elements
//    whose full (value, id) key beats T are pushed, with ballot + mbcnt, into a single-producer
//    ring in LDS.
//  * The fourth wave is the consumer: it drains the rings, keeps the one sorted list of the
//    row's K best keys in registers (one key per lane, insertion by DPP lane shift, or a bitonic
//    sort + merge for large batches) and publishes the list's K-th key as the new threshold. The
//    serial list work thus never stalls the HBM stream. Each producer seeds the threshold from
//    its first tile with the K-th largest lane maximum (radix select across lanes).
//  * Rows split over several workgroups (small N*B) write partial results to the workspace and a
//    second kernel merges them.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "common.hpp"
#include "lilicorr.h"

namespace lilicorr {
namespace {

constexpr float kLog2eF = 1.44269504088896340736f;  // log2(e) rounded to fp32
constexpr int kPerLane = 32;                         // elements per lane per tile
constexpr int kRebase = 16;                          // max term exponent before the reference moves
constexpr int kTopkWaves = 4;                        // wave 0 consumes, waves 1..3 produce
constexpr int kProducers = kTopkWaves - 1;
constexpr uint32_t kRing = 512;                      // keys per producer ring (power of two)
constexpr int kSpinLimit = 1 << 22;                  // bound on any wait (never reached)

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

struct TopkShared {
  uint64_t T;                      // best published threshold key (atomic max)
  uint32_t tail[kProducers];       // ring write positions (producer-owned)
  uint32_t head[kProducers];       // ring read positions (consumer-owned)
  uint32_t done;                   // producers finished
  int cref[kProducers];
  int cvalid[kProducers];
  float s[kProducers];
  uint64_t ring[kProducers][kRing];
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
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const uint32_t off = (uint32_t)((rel_chunk0 + (int64_t)u * kWave + lane) * 16);
    // cache policy 3 (sc0 nt): streaming data, read once (measured fastest for this pass)
    raw[u] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rsrc, off, 0, 3));
  }
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

// 1 if the tile may hold an element >= Tv (> Tv when strict), for a positive bf16-representable
// Tv: positive bf16 bit patterns order like signed 16-bit integers, and every negative pattern
// (including the -inf padding) is below them. Packed 16-bit max over the raw tile.
template <bool STRICT>
__device__ __forceinline__ int bf16_screen(const u32x4 (&raw)[4], float Tv) {
  // (each dword is copied to a scalar before the bit cast: a bit cast applied directly to a
  // vector element subscript has been seen to read element 0)
  const uint32_t w00 = raw[0][0];
  i16x2 m = __builtin_bit_cast(i16x2, w00);
#pragma unroll
  for (int u = 0; u < 4; ++u)
#pragma unroll
    for (int q = 0; q < 4; ++q)
      if (u || q) {
        const uint32_t w = raw[u][q];
        m = __builtin_elementwise_max(m, __builtin_bit_cast(i16x2, w));
      }
  const int mx = m[0] > m[1] ? (int)m[0] : (int)m[1];
  const int tb = (int)(__float_as_uint(Tv) >> 16);
  return STRICT ? (mx > tb ? 1 : 0) : (mx >= tb ? 1 : 0);
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
};

__device__ __forceinline__ void rebase(Producer& pr, int need) {
  if (!pr.cvalid) {
    pr.cref = need;
    pr.cvalid = 1;
  } else if (need - pr.cref > kRebase) {
    pr.s = ldexpf(pr.s, pr.cref - need);
    pr.cref = need;
  }
}

// Append the keys of the lanes with `live` set to this producer's ring.
__device__ __forceinline__ void push_keys(Producer& pr, TopkShared& sh, uint64_t key, bool live) {
  const uint64_t m = __ballot(live);
  if (!m) return;
  const uint32_t n = (uint32_t)__popcll(m);
  if (pr.tail + n - pr.head > kRing) {
    // make everything written so far visible to the consumer before waiting for it
    if (lane_id() == 0)
      __hip_atomic_store(&sh.tail[pr.p], pr.tail, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
    for (int spin = 0; spin < kSpinLimit; ++spin) {
      pr.head = uniform32(__hip_atomic_load(&sh.head[pr.p], __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP));
      if (pr.tail + n - pr.head <= kRing) break;
      __builtin_amdgcn_s_sleep(1);
    }
  }
  if (live) {
    const uint32_t off = __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
    sh.ring[pr.p][(pr.tail + off) & (kRing - 1)] = key;
  }
  pr.tail += n;
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

// Push every element of the tile whose key beats T, scanning only the 8-element blocks that reach
// tv (strict: x > tv, else x >= tv; see strict_ok).
template <bool STRICT, int NE, typename IdOf, typename ValidOf>
__device__ __forceinline__ void push_tile(Producer& pr, TopkShared& sh, const float (&x)[NE],
                                          IdOf id_of, ValidOf valid_of, float tv, uint64_t T) {
  constexpr int NB = (NE + 7) / 8;
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    float bm = -__builtin_inff();
#pragma unroll
    for (int j = 8 * b; j < 8 * b + 8 && j < NE; ++j) bm = fmaxf(bm, x[j]);
    if (!__ballot(STRICT ? (bm > tv) : (bm >= tv))) continue;
#pragma unroll
    for (int j = 8 * b; j < 8 * b + 8 && j < NE; ++j) {
      const bool pred = STRICT ? (x[j] > tv) : (x[j] >= tv);
      if (!__ballot(pred)) continue;
      const uint64_t kj = make_key(x[j], id_of(j));
      push_keys(pr, sh, kj, pred && valid_of(j) && kj > T);
    }
  }
}

// One tile of NE elements per lane. x[] are the values; id_of(j) gives the row-relative token id
// of element j of this lane and valid_of(j) whether it is a real element (tiles are padded with
// -inf). raw, when not null, is the tile's raw bf16 data for the packed screen; tile_min_id is
// the smallest id in the tile (0: never screen strictly).
template <int NE, typename IdOf, typename ValidOf>
__device__ __forceinline__ void produce_tile(Producer& pr, TopkShared& sh, const float (&x)[NE],
                                             const u32x4* raw, IdOf id_of, ValidOf valid_of, int K,
                                             bool first, uint32_t tile_min_id) {
  const int lane = lane_id();
  uint64_t T = atomic_load_T(sh);
  if (pr.seedT > T) T = pr.seedT;
  float lane_max = -__builtin_inff();
  bool have_max = false;
  if (first) {
#pragma unroll
    for (int j = 0; j < NE; ++j) lane_max = fmaxf(lane_max, x[j]);
    have_max = true;
    const uint64_t seedT = uniform64(seed_threshold(lane_max, K));
    if (key_value(seedT) > -__builtin_inff() && seedT > T) {
      // a bound for the whole row: the K lanes behind it hold K distinct elements at or above it
      pr.seedT = seedT;
      T = seedT;
      publish_T(sh, seedT);
    }
  }
  const float tv = key_value(T);
  const bool strict = strict_ok(T, tile_min_id);
  int flag;
  if (raw != nullptr && !first && tv > 0.f) {
    const u32x4(&r4)[4] = *reinterpret_cast<const u32x4(*)[4]>(raw);
    flag = strict ? bf16_screen<true>(r4, tv) : bf16_screen<false>(r4, tv);
  } else {
    if (!have_max) {
#pragma unroll
      for (int j = 0; j < NE; ++j) lane_max = fmaxf(lane_max, x[j]);
      have_max = true;
    }
    flag = strict ? (lane_max > tv) : (lane_max >= tv);
  }

  if (__ballot(flag != 0)) {
    if (strict)
      push_tile<true>(pr, sh, x, id_of, valid_of, tv, T);
    else
      push_tile<false>(pr, sh, x, id_of, valid_of, tv, T);
    if (lane == 0)
      __hip_atomic_store(&sh.tail[pr.p], pr.tail, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
  }

  // Exp sums. The reference follows the threshold value (an element's value, so never above the
  // row maximum); an element far above it shows up as a tile sum beyond 2^kBig (or inf), and the
  // tile is then summed again with the reference at the tile maximum.
  if (tv > -__builtin_inff()) rebase(pr, ref_for(tv));
  if (!pr.cvalid) {
    if (!have_max) {
#pragma unroll
      for (int j = 0; j < NE; ++j) lane_max = fmaxf(lane_max, x[j]);
      have_max = true;
    }
    const float m = wave_max_dpp(lane_max);
    if (m > -__builtin_inff()) rebase(pr, ref_for(m));
  }
  if (pr.cvalid) {
    float sum = tile_exp_sum(x, pr.cref);
    if (__ballot(!(sum <= kBig))) {
      if (!have_max) {
#pragma unroll
        for (int j = 0; j < NE; ++j) lane_max = fmaxf(lane_max, x[j]);
      }
      const int need = ref_for(wave_max_dpp(lane_max));
      if (need > pr.cref) {
        pr.s = ldexpf(pr.s, pr.cref - need);
        pr.cref = need;
      }
      sum = tile_exp_sum(x, pr.cref);
    }
    pr.s += sum;
  }
}

// ---- consumer ---------------------------------------------------------------------------------

struct Consumer {
  uint64_t L;      // this lane's entry of the sorted list (lanes >= K hold 0)
  uint64_t T_own;  // (u) key of the list's K-th entry, 0 while the list is not full
};

// Merge a batch of up to 64 keys (one per lane, 0 = none) into the list.
__device__ __forceinline__ void consume_batch(Consumer& c, TopkShared& sh, uint64_t v, int K) {
  const int lane = lane_id();
  uint64_t T = atomic_load_T(sh);
  if (c.T_own > T) T = c.T_own;
  uint64_t m = __ballot(v > T);
  if (!m) return;
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

__device__ __forceinline__ void consume_all(Consumer& c, TopkShared& sh, int K) {
  const int lane = lane_id();
  uint32_t head[kProducers];
#pragma unroll
  for (int p = 0; p < kProducers; ++p) head[p] = 0;
  for (int idle = 0; idle < kSpinLimit;) {
    bool any = false;
#pragma unroll
    for (int p = 0; p < kProducers; ++p) {
      const uint32_t t = uniform32(__hip_atomic_load(&sh.tail[p], __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP));
      while (head[p] != t) {
        const uint32_t n = t - head[p] < (uint32_t)kWave ? t - head[p] : (uint32_t)kWave;
        const uint64_t v = (uint32_t)lane < n ? sh.ring[p][(head[p] + lane) & (kRing - 1)] : 0ull;
        head[p] += n;
        if (lane == 0)
          __hip_atomic_store(&sh.head[p], head[p], __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
        consume_batch(c, sh, v, K);
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
      if (!more) break;
      continue;
    }
    __builtin_amdgcn_s_sleep(2);
    ++idle;
  }
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
    float* __restrict__ logp, float* __restrict__ feat, unsigned char* __restrict__ partials) {
  constexpr int EPC = ElemTraits<BF16>::kEPC;
  constexpr int U = kPerLane / EPC;
  constexpr int TILE = U * kWave;  // chunks per wave tile

  __shared__ TopkShared sh;

  const int lane = lane_id();
  const int wave = threadIdx.x / kWave;
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
    consume_all(cons, sh, K);
  } else {
    Producer pr;
    pr.p = wave - 1;
    pr.seedT = 0;
    pr.tail = 0;
    pr.head = 0;
    pr.cref = 0;
    pr.cvalid = 0;
    pr.s = 0.f;
    // producer p streams tiles p, p + 3, p + 6, ... (the workgroup reads one contiguous window
    // at a time); its tiles come in increasing id order
    const uint32_t body_end_id = (uint32_t)(c_end * EPC - rowbase);
    bool first = true;
    auto process = [&](u32x4 (&raw)[U], int64_t t) {
      if ((t + 1) * TILE > nchunks) pad_tile<BF16>(raw, t * TILE, nchunks);
      float x[kPerLane];
      unpack_tile<BF16>(raw, x);
      const int64_t tc0 = c_beg + t * TILE;
      const uint32_t tile_min_id = (uint32_t)(tc0 * EPC - rowbase);
      // id of element j of this lane: the per-lane base is made opaque to the optimiser, which
      // would otherwise keep all 32 (lane, j) offsets live across the loop
      uint32_t lane_base = tile_min_id + (uint32_t)(lane * EPC);
      __asm__ volatile("" : "+v"(lane_base));
      auto id_of = [&](int j) -> uint32_t {
        return lane_base + (uint32_t)((j / EPC) * kWave * EPC + (j % EPC));
      };
      auto valid_of = [&](int j) -> bool { return id_of(j) < body_end_id; };
      produce_tile<kPerLane>(pr, sh, x, BF16 ? raw : nullptr, id_of, valid_of, K, first, tile_min_id);
      first = false;
    };
    // one tile in flight: the next tile's loads are issued (unconditionally: past the segment end
    // the bounded descriptor returns zeros without touching memory) before the current tile is
    // processed
    u32x4 raw[U];
    load_tile<BF16>(raw, rsrc, (int64_t)pr.p * TILE);
    for (int64_t t = pr.p; t < ntiles; t += kProducers) {
      u32x4 cur[U];
#pragma unroll
      for (int u = 0; u < U; ++u) cur[u] = raw[u];
      load_tile<BF16>(raw, rsrc, (t + kProducers) * TILE);
      process(cur, t);
    }
    if (wave == kTopkWaves - 1 && n_head + n_tail > 0) {
      // ragged head/tail elements, one per lane
      float x1[1];
      int64_t g = -1;
      if (lane < n_head) g = g0 + lane;
      else if (lane < n_head + n_tail) g = c_end * EPC + (lane - n_head);
      if (g >= 0) {
        x1[0] = BF16 ? __uint_as_float((uint32_t)reinterpret_cast<const uint16_t*>(logits)[g] << 16)
                     : reinterpret_cast<const float*>(logits)[g];
      } else {
        x1[0] = -__builtin_inff();
      }
      auto id_of1 = [&](int) -> uint32_t { return (uint32_t)(g - rowbase); };
      auto valid_of1 = [&](int) -> bool { return g >= 0; };
      // head ids precede the body: never screen strictly here
      produce_tile<1>(pr, sh, x1, nullptr, id_of1, valid_of1, K, first, 0u);
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

// One wave per row: merge the `split` partial results of the row.
__global__ __launch_bounds__(kWave) void topk_merge_kernel(const unsigned char* __restrict__ partials,
                                                         int K, int split, int32_t* __restrict__ ids,
                                                         float* __restrict__ logp,
                                                         float* __restrict__ feat) {
  const int lane = lane_id();
  const int64_t row = blockIdx.x;
  uint64_t merged = 0;
  int C = 0, any = 0;
  for (int p = 0; p < split; ++p) {
    const unsigned char* q = partials + ((size_t)row * split + p) * partial_stride(K);
    const Partial* hdr = reinterpret_cast<const Partial*>(q);
    if (hdr->cvalid) {
      C = any ? (hdr->cref > C ? hdr->cref : C) : hdr->cref;
      any = 1;
    }
  }
  float S = 0.f;
  for (int p = 0; p < split; ++p) {
    const unsigned char* q = partials + ((size_t)row * split + p) * partial_stride(K);
    const Partial* hdr = reinterpret_cast<const Partial*>(q);
    const uint64_t* keys = reinterpret_cast<const uint64_t*>(q + sizeof(Partial));
    if (hdr->cvalid) S += ldexpf(hdr->s, hdr->cref - C);
    uint64_t k = lane < K ? keys[lane] : 0ull;
    merged = p == 0 ? k : merge_desc64(merged, k);
  }
  write_row(merged, (log2((double)S) + (double)C) / (double)kLog2eF, row, K, ids, logp, feat);
}

// Number of workgroups per row: enough workgroups to fill the chip (about four per CU), but
// no segment shorter than two workgroup tiles.
int topk_split(int64_t rows, int64_t V, bool bf16) {
  const int64_t wg_tile = (int64_t)kProducers * kWave * kPerLane;
  const int64_t target = 1024;
  int64_t by_fill = (target + rows - 1) / rows;
  int64_t by_len = V / (2 * wg_tile);
  int64_t s = by_fill < by_len ? by_fill : by_len;
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

extern "C" size_t lilicorr_topk_workspace_bytes(int64_t N, int64_t B, int64_t V, int K) {
  if (!topk_args_ok(N, B, V, K) || K > 64 || K > V) return 0;
  int split = topk_split(N * B, V, true);
  if (split == 1) return 0;
  return (size_t)(N * B) * split * partial_stride(K);
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
  const size_t need = split == 1 ? 0 : (size_t)rows * split * partial_stride(K);
  if (need > 0 && (!workspace || workspace_bytes < need)) return LILICORR_ERR_WORKSPACE;
  if (need > 0 && !aligned16(workspace)) return LILICORR_ERR_ALIGNMENT;
  if (rows * split > 0x7fffffffll) return LILICORR_ERR_UNSUPPORTED;

  dim3 grid((unsigned)(rows * split)), block(kTopkWaves * kWave);
  unsigned char* ws = static_cast<unsigned char*>(workspace);
  if (bf16)
    hipLaunchKernelGGL(topk_lse_kernel<true>, grid, block, 0, stream, logits, V, K, split, ids, logp,
                       feat, ws);
  else
    hipLaunchKernelGGL(topk_lse_kernel<false>, grid, block, 0, stream, logits, V, K, split, ids,
                       logp, feat, ws);
  if (launch_status() != LILICORR_OK) return LILICORR_ERR_HIP;
  if (split > 1) {
    hipLaunchKernelGGL(topk_merge_kernel, dim3((unsigned)rows), dim3(kWave), 0, stream, ws, K, split,
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
