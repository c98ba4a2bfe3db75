// Step 1 of the path: vocabulary-wide log-normalisation fused with exact top-K selection
// (Sec. 3.2 candidate pool; implementation appendix, "Serving": normalisation and candidate
// extraction in one kernel).
//
// Design (gfx950):
//  * The logits are streamed from HBM exactly once with 16-byte non-temporal loads; each wave
//    owns interleaved tiles of 64 lanes x 32 elements (4 KB of bf16) of one row segment.
//  * Log-sum-exp: every element adds exp2(x*log2e - c) to a per-lane partial sum; c is a
//    wave-uniform integer reference (log2 units), so moving it only rescales the partial sums by
//    an exact power of two. c is raised only on the rare tiles that hold a new candidate, which
//    keeps every term below 2^17 and the running maximum's term at or above 2^-1.
//  * Top-K: each wave keeps its K best (value, id) keys in registers, one per lane, sorted.
//    A wave-uniform threshold (the K-th key of this wave or of any wave of the workgroup, shared
//    through LDS) filters the tile: bf16 tiles are screened with packed 16-bit integer max on the
//    raw bit patterns, so a tile with no candidate costs about half an instruction per element.
//    Candidates are inserted one at a time with a DPP lane shift. The first tile of each wave
//    seeds the threshold with the K-th largest lane maximum (bitonic sort across lanes).
//  * Waves of a workgroup merge their lists with bitonic merges in LDS. Rows split over several
//    workgroups (small N*B) write partial results to the workspace and a second kernel merges.
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
constexpr int kTopkWaves = 4;

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

// Per-wave running state. Scalars marked (u) are wave-uniform.
struct WaveTopk {
  uint64_t L;      // this lane's entry of the sorted list (lanes >= K hold 0)
  uint64_t T_own;  // (u) key of this wave's K-th entry, 0 while the list is not full
  uint64_t T;      // (u) reject threshold: max(T_own, workgroup-shared threshold)
  float Tv;        // (u) value part of T (-inf for T == 0)
  int cref;        // (u) log2-units reference of the exp sums
  int cvalid;      // (u) cref is set
  float s;         // per-lane partial sum of exp2(x*log2e - cref)
};

__device__ __forceinline__ void set_threshold(WaveTopk& w, uint64_t shared_T) {
  uint64_t t = w.T_own > shared_T ? w.T_own : shared_T;
  w.T = uniform64(t);
  w.Tv = key_value(w.T);
}

__device__ __forceinline__ void insert_key(WaveTopk& w, uint64_t key, int K, uint64_t shared_T) {
  const int lane = lane_id();
  int pos = __popcll(__ballot(w.L > key));
  uint64_t up = shift_up64(w.L);
  uint64_t nl = lane < pos ? w.L : (lane == pos ? key : up);
  w.L = lane < K ? nl : 0ull;
  w.T_own = readlane64(w.L, K - 1);
  set_threshold(w, shared_T);
}

__device__ __forceinline__ void rebase(WaveTopk& w, int need) {
  if (!w.cvalid) {
    w.cref = need;
    w.cvalid = 1;
  } else if (need - w.cref > kRebase) {
    w.s = ldexpf(w.s, w.cref - need);
    w.cref = need;
  }
}

__device__ __forceinline__ int ref_for(float v) { return (int)ceilf(v * kLog2eF); }

// Process one tile of NE elements per lane. x[] are the values; id_of(j, lane) gives the
// row-relative token id of element j of `lane`. `flag_in` carries a per-lane flag computed by a
// cheaper screen (or -1 to screen here with float compares).
template <int NE, typename IdOf>
__device__ __forceinline__ void process_tile(WaveTopk& w, const float (&x)[NE], IdOf id_of, int K,
                                             bool first, int flag_in, uint64_t* sh_T) {
  uint64_t shared_T = uniform64(__hip_atomic_load(sh_T, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP));
  set_threshold(w, shared_T);

  float lane_max = -__builtin_inff();
  if (first || flag_in < 0) {
#pragma unroll
    for (int j = 0; j < NE; ++j) lane_max = fmaxf(lane_max, x[j]);
  }
  if (first) {
    // seed: the K-th largest lane maximum bounds the K-th largest element from below
    float sorted = sort_desc64(lane_max);
    float seed = readlanef(sorted, K - 1);
    uint64_t seedT = (uint64_t)order_bits(seed) << 32;
    if (seed > -__builtin_inff() && seedT > shared_T) {
      shared_T = seedT;
      // a bound for the whole row: publish it to the other waves of the workgroup
      if (lane_id() == 0) atomicMax((unsigned long long*)sh_T, (unsigned long long)seedT);
    }
    set_threshold(w, shared_T);
  }
  bool flag = (flag_in < 0 || first) ? (lane_max >= w.Tv) : (flag_in != 0);

  float cmax = -__builtin_inff();
  if (__ballot(flag)) {
#pragma unroll
    for (int j = 0; j < NE; ++j) {
      uint64_t m = __ballot(x[j] >= w.Tv);
      while (m) {
        int ln = __ffsll((long long)m) - 1;
        m &= m - 1;
        float v = readlanef(x[j], ln);
        cmax = fmaxf(cmax, v);
        uint64_t key = make_key(v, id_of(j, ln));
        if (key > w.T) insert_key(w, key, K, shared_T);
      }
    }
    if (w.T_own > shared_T && lane_id() == 0)
      atomicMax((unsigned long long*)sh_T, (unsigned long long)w.T_own);
  }
  // keep every term of this tile below 2^(kRebase+1): non-candidates are below Tv, candidates
  // at most cmax
  float ref = fmaxf(cmax, w.Tv);
  if (ref > -__builtin_inff()) rebase(w, ref_for(ref));
  if (w.cvalid) {
    const float c = -(float)w.cref;
    float t[NE];
#pragma unroll
    for (int j = 0; j < NE; ++j) t[j] = __builtin_amdgcn_exp2f(fmaf(x[j], kLog2eF, c));
#pragma unroll
    for (int span = 1; span < NE; span <<= 1)
#pragma unroll
      for (int j = 0; j + span < NE; j += 2 * span) t[j] += t[j + span];
    w.s += t[0];
  }
}

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef short i16x2 __attribute__((ext_vector_type(2)));

template <bool BF16>
__device__ __forceinline__ void load_tile(u32x4 (&raw)[kPerLane / ElemTraits<BF16>::kEPC],
                                          const u32x4* __restrict__ chunks, int64_t c0,
                                          int64_t c_end) {
  constexpr int U = kPerLane / ElemTraits<BF16>::kEPC;
  const u32x4 pad = BF16 ? u32x4{0xFF80FF80u, 0xFF80FF80u, 0xFF80FF80u, 0xFF80FF80u}
                         : u32x4{0xFF800000u, 0xFF800000u, 0xFF800000u, 0xFF800000u};
  const int lane = lane_id();
#pragma unroll
  for (int u = 0; u < U; ++u) {
    int64_t c = c0 + (int64_t)u * kWave + lane;
    raw[u] = c < c_end ? __builtin_nontemporal_load(chunks + c) : pad;
  }
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

// 1 if any bf16 element of the tile is >= Tv, for a positive bf16-representable Tv: positive
// bf16 bit patterns order like signed 16-bit integers and every negative pattern is below them.
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
  int mx = m[0] > m[1] ? (int)m[0] : (int)m[1];
  int tb = (int)(__float_as_uint(Tv) >> 16);
  return mx >= tb ? 1 : 0;
}

template <bool BF16>
__global__ __launch_bounds__(kTopkWaves * kWave) void topk_lse_kernel(
    const void* __restrict__ logits, int64_t V, int K, int split, int32_t* __restrict__ ids,
    float* __restrict__ logp, unsigned char* __restrict__ partials) {
  constexpr int EPC = ElemTraits<BF16>::kEPC;
  constexpr int U = kPerLane / EPC;
  constexpr int TILE = U * kWave;  // chunks per wave tile

  __shared__ uint64_t sh_T;
  __shared__ uint64_t sh_list[kTopkWaves][kWave];
  __shared__ int sh_cref[kTopkWaves];
  __shared__ int sh_cvalid[kTopkWaves];
  __shared__ float sh_s[kTopkWaves];

  const int lane = lane_id();
  const int wave = threadIdx.x / kWave;
  const int64_t row = blockIdx.x / split;
  const int part = blockIdx.x % split;
  const int64_t rowbase = row * V;
  const int64_t span = (V + split - 1) / split;
  const int64_t g0 = rowbase + (int64_t)part * span;
  const int64_t g1 = rowbase + ((int64_t)(part + 1) * span < V ? (int64_t)(part + 1) * span : V);

  if (threadIdx.x == 0) sh_T = 0;
  __syncthreads();

  WaveTopk w;
  w.L = 0;
  w.T_own = 0;
  w.T = 0;
  w.Tv = -__builtin_inff();
  w.cref = 0;
  w.cvalid = 0;
  w.s = 0.f;

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
  const u32x4* chunks = reinterpret_cast<const u32x4*>(logits);

  bool first = true;
  int64_t t = wave;
  u32x4 raw[U];
  if (t < ntiles) load_tile<BF16>(raw, chunks, c_beg + t * TILE, c_end);
  for (; t < ntiles; t += kTopkWaves) {
    u32x4 cur[U];
#pragma unroll
    for (int u = 0; u < U; ++u) cur[u] = raw[u];
    if (t + kTopkWaves < ntiles) load_tile<BF16>(raw, chunks, c_beg + (t + kTopkWaves) * TILE, c_end);
    float x[kPerLane];
    unpack_tile<BF16>(cur, x);
    const int64_t tc0 = c_beg + t * TILE;
    auto id_of = [&](int j, int ln) -> uint32_t {
      int64_t c = tc0 + (int64_t)(j / EPC) * kWave + ln;
      return (uint32_t)(c * EPC + (j % EPC) - rowbase);
    };
    int flag = -1;
    if (BF16 && !first) {
      uint64_t st = uniform64(__hip_atomic_load(&sh_T, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP));
      uint64_t tt = w.T_own > st ? w.T_own : st;
      float tv = key_value(tt);
      if (tv > 0.f) flag = bf16_screen(reinterpret_cast<const u32x4(&)[4]>(cur), tv);
    }
    process_tile<kPerLane>(w, x, id_of, K, first, flag, &sh_T);
    first = false;
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
    auto id_of1 = [&](int, int ln) -> uint32_t {
      int64_t gg = ln < n_head ? g0 + ln : c_end * EPC + (ln - n_head);
      return (uint32_t)(gg - rowbase);
    };
    process_tile<1>(w, x1, id_of1, K, first, -1, &sh_T);
  }

  // merge the waves of this workgroup
  sh_list[wave][lane] = w.L;
  float ws = wave_sum(w.s);
  if (lane == 0) {
    sh_cref[wave] = w.cref;
    sh_cvalid[wave] = w.cvalid;
    sh_s[wave] = ws;
  }
  __syncthreads();
  if (wave != 0) return;

  int C = 0, any = 0;
  for (int i = 0; i < kTopkWaves; ++i)
    if (sh_cvalid[i]) {
      C = any ? (sh_cref[i] > C ? sh_cref[i] : C) : sh_cref[i];
      any = 1;
    }
  float S = 0.f;
  for (int i = 0; i < kTopkWaves; ++i)
    if (sh_cvalid[i]) S += ldexpf(sh_s[i], sh_cref[i] - C);
  uint64_t merged = sh_list[0][lane];
  for (int i = 1; i < kTopkWaves; ++i) merged = merge_desc64(merged, sh_list[i][lane]);

  if (split == 1) {
    if (lane < K) {
      double lse = (log2((double)S) + (double)C) / (double)kLog2eF;
      ids[row * K + lane] = (int32_t)key_id(merged);
      logp[row * K + lane] = (float)((double)key_value(merged) - lse);
    }
  } else {
    unsigned char* p = partials + ((size_t)row * split + part) * partial_stride(K);
    Partial* hdr = reinterpret_cast<Partial*>(p);
    uint64_t* keys = reinterpret_cast<uint64_t*>(p + sizeof(Partial));
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
                                                         float* __restrict__ logp) {
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
  if (lane < K) {
    double lse = (log2((double)S) + (double)C) / (double)kLog2eF;
    ids[row * K + lane] = (int32_t)key_id(merged);
    logp[row * K + lane] = (float)((double)key_value(merged) - lse);
  }
}

// Number of workgroups per row: enough workgroups to fill the chip (about four per CU), but
// no segment shorter than two workgroup tiles.
int topk_split(int64_t rows, int64_t V, bool bf16) {
  const int64_t wg_tile = (int64_t)kTopkWaves * kWave * kPerLane;
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

extern "C" lilicorr_status lilicorr_topk(const void* logits, lilicorr_dtype dtype, int64_t N,
                                         int64_t B, int64_t V, int K, int32_t* ids, float* logp,
                                         void* workspace, size_t workspace_bytes,
                                         hipStream_t stream) {
  if (!logits || !ids || !logp) return LILICORR_ERR_INVALID_ARG;
  if (dtype != LILICORR_F32 && dtype != LILICORR_BF16) return LILICORR_ERR_INVALID_ARG;
  if (!topk_args_ok(N, B, V, K)) return LILICORR_ERR_INVALID_ARG;
  if (K > 64 || K > V) return LILICORR_ERR_UNSUPPORTED;
  if (!aligned16(logits) || !aligned16(ids) || !aligned16(logp)) return LILICORR_ERR_ALIGNMENT;
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
    hipLaunchKernelGGL(topk_lse_kernel<true>, grid, block, 0, stream, logits, V, K, split, ids, logp, ws);
  else
    hipLaunchKernelGGL(topk_lse_kernel<false>, grid, block, 0, stream, logits, V, K, split, ids, logp, ws);
  if (launch_status() != LILICORR_OK) return LILICORR_ERR_HIP;
  if (split > 1) {
    hipLaunchKernelGGL(topk_merge_kernel, dim3((unsigned)rows), dim3(kWave), 0, stream, ws, K, split, ids, logp);
    if (launch_status() != LILICORR_OK) return LILICORR_ERR_HIP;
  }
  return LILICORR_OK;
}
