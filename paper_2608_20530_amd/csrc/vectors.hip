// Step 2 of the path: candidate in/out vectors. The head's two linear heads emit an out and an in
// vector per candidate, each normalised to unit norm (Sec. 3.2, implementation appendix); here
// they are u = E[id] W (W[i][j], row-vector convention) followed by v = u / ||u||.
//
// bf16 embeddings: a dense [M x d] x [d x d] contraction per side, run on the bf16 matrix cores
// (v_mfma_f32_16x16x32_bf16). Every fp32 weight is split exactly into three bf16 terms
// (hi + mid + lo == w), so each bf16 x bf16 product is exact in fp32 and the fp32 accumulation
// gives fp32-grade results at three times the MFMA work. A workgroup owns a tile of candidate rows
// and all d columns of one side, so the L2 norm of every row is finished in-kernel. The gathered
// embedding rows (the A operand) are staged once in LDS; each wave owns four 16-column blocks and
// streams their B fragments (three terms each) from the L2-resident packed weights through two
// register buffers, loading k-block kb+1 while the MFMAs of kb run. The packed layout is padded to
// whole wave column groups and an even number of k-blocks, so the MFMA loop has no branches.
// The vectors are written with non-temporal stores: they are read once, by the pair-score pass,
// and at the stress width (537 MB) stores that stay in the caches are written back while that
// pass reads (measured at N=256, K=32, d=512: 511 -> 489 us here, 134 -> 102 us for the pair
// scores that follow).
//
// fp32 embeddings: products are no longer exact in bf16, so a plain fp32 FMA kernel is used.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "common.hpp"
#include "lilicorr.h"
#include "projection.hpp"

namespace lilicorr {
namespace {

__device__ __forceinline__ uint16_t split_term(float w, int term) {
  float hi = __uint_as_float(__float_as_uint(w) & 0xffff0000u);
  float r1 = w - hi;  // exact: the low 16 significand bits of w
  float mid = __uint_as_float(__float_as_uint(r1) & 0xffff0000u);
  float r2 = r1 - mid;  // exact, at most 8 significant bits: a bf16 value
  float t = term == 0 ? hi : (term == 1 ? mid : r2);
  return (uint16_t)(__float_as_uint(t) >> 16);
}

__global__ void pack_weights_kernel(const float* __restrict__ W_in, const float* __restrict__ W_out,
                                    int d, int nbp, int dkp, uint16_t* __restrict__ frags,
                                    float* __restrict__ f32copy) {
  const int64_t nfrag = (int64_t)2 * dkp * 3 * nbp * 512;
  const int64_t ncopy = (int64_t)2 * d * d;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < nfrag + ncopy;
       i += (int64_t)gridDim.x * blockDim.x) {
    if (i < nfrag) {
      int64_t r = i;
      const int e = (int)(r % 8); r /= 8;
      const int lane = (int)(r % 64); r /= 64;
      const int nb = (int)(r % nbp); r /= nbp;
      const int term = (int)(r % 3); r /= 3;
      const int kb = (int)(r % dkp); r /= dkp;
      const int side = (int)r;
      const int k = kb * 32 + (lane / 16) * 8 + e;
      const int col = nb * 16 + lane % 16;
      const float* W = side == 0 ? W_in : W_out;
      const float w = (k < d && col < d) ? W[(int64_t)k * d + col] : 0.f;
      frags[i] = split_term(w, term);
    } else {
      const int64_t j = i - nfrag;
      const int side = (int)(j / ((int64_t)d * d));
      const int64_t off = j % ((int64_t)d * d);
      f32copy[j] = (side == 0 ? W_in : W_out)[off];
    }
  }
}

// One workgroup: RM*16 candidate rows x all d columns of one side. The gathered embedding rows
// (the A operand) are staged once in LDS; wave w owns column blocks [4w, 4w+4). Each B fragment
// feeds RM MFMAs and each A fragment 12.
template <int RM, int MAXT>
__global__ __launch_bounds__(MAXT) void cand_vectors_mfma_kernel(
    const int32_t* __restrict__ ids, const uint16_t* __restrict__ E,
    const unsigned char* __restrict__ frags, int64_t M, int64_t V, int d, int nbp, int dkp,
    float* __restrict__ in_vec, float* __restrict__ out_vec) {
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  constexpr int ROWS = RM * 16;
  const int dpad = dkp * 32;
  const int astride = dpad + 8;  // bf16 elements per LDS row (16-byte multiple, spreads banks)
  const int side = blockIdx.y;
  const int nthreads = blockDim.x;
  const int nwaves = nthreads / kWave;
  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int wave = tid / kWave;
  const int64_t row0 = blockIdx.x * (int64_t)ROWS;

  uint16_t* A = reinterpret_cast<uint16_t*>(smem);  // [ROWS][astride]
  float* ssbuf = reinterpret_cast<float*>(smem + (size_t)ROWS * astride * 2);  // [nwaves][ROWS]
  int32_t* rid = reinterpret_cast<int32_t*>(ssbuf + nwaves * ROWS);             // [ROWS]

  // this wave's fragments: column blocks [4 wave, 4 wave + 4) of one (k-block, term) slice
  const size_t slice = (size_t)nbp * 1024;
  const unsigned char* wf =
      frags + (size_t)side * dkp * 3 * slice + (size_t)wave * kNbPerWave * 1024 + lane * 16;
  BFrag<kNbPerWave> b0;
  load_bfrag<kNbPerWave>(b0, wf, slice, 0);  // in flight during the gather

  // gather the embedding rows (zero rows past M or for ids outside [0, V); zero k-padding)
  for (int r = tid; r < ROWS; r += nthreads) {
    const int64_t row = row0 + r;
    const int32_t id = row < M ? ids[row] : -1;
    rid[r] = (id >= 0 && id < V) ? id : -1;
  }
  __syncthreads();
  gather_rows(A, astride, ROWS, rid, E, d, dpad, tid, nthreads);
  __syncthreads();

  f32x4 acc[RM][kNbPerWave];
  if constexpr (MAXT > 512) {
    (void)b0;  // the 1024-thread instance streams its weights one column block at a time
    project_tile_lean<RM>(acc, A, astride, wf, slice, dkp, lane);
  } else {
    project_tile<RM, kNbPerWave>(acc, b0, A, astride, wf, slice, dkp, lane);
  }
  row_sumsq<RM, kNbPerWave>(acc, ssbuf + wave * ROWS, lane);
  __syncthreads();
  float* out = side == 0 ? in_vec : out_vec;
  const int col0 = wave * kNbPerWave * 16 + (lane & 15);
#pragma unroll
  for (int mb = 0; mb < RM; ++mb) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int rl = mb * 16 + (lane >> 4) * 4 + i;
      float tot = 0.f;
      for (int g = 0; g < nwaves; ++g) tot += ssbuf[g * ROWS + rl];
      const float inv = tot > 0.f ? 1.0f / sqrtf(tot) : 0.f;
      const int64_t r = row0 + rl;
      if (r < M) {
#pragma unroll
        for (int nb = 0; nb < kNbPerWave; ++nb)
          if (col0 + nb * 16 < d)
            __builtin_nontemporal_store(acc[mb][nb][i] * inv, &out[r * d + col0 + nb * 16]);
      }
    }
  }
}

typedef __attribute__((address_space(3))) void* lds_ptr_t;

// Wide persistent variant for many tiles at 448 < d <= 512 (32 k-blocks of the contraction, 32
// column blocks). The weight fragments stream from L2 once per tile and are reused by every row
// of it, so the L2 read per row falls with the tile height; at 64 rows the fragment read keeps
// pace with the matrix cores only just. Here a tile is 128 rows and each of eight waves (two per
// SIMD, 256 registers each) owns 64 columns: its 128 x 64 accumulator block sits in ordinary
// registers, where the matrix cores run faster than from the accumulation registers (a
// register-only probe of this loop shape: 1.98 against 1.1-1.7 PFLOP/s).
//  * The gathered tile (128 rows of bf16, both halves of the k range) lives in LDS as
//    [half][row][256 bf16 + 8 of padding], so the 16 rows one fragment read touches fall in 16
//    different bank groups and every k-block's reads sit at fixed offsets from one lane base.
//  * Rows arrive by direct global-to-LDS loads, one half row per wave instruction (32 lanes),
//    two per wave in every k-block: a tile's second half while its first half is multiplied,
//    the next tile's first half while its second half is. The ids of a wave's 16 rows sit one
//    per lane, so a copy reads no LDS in the k-loop.
//  * The k-block loop is unrolled, so the accumulators stay in place across k-blocks, and the
//    weight fragments come through a buffer descriptor with one lane offset (their k-block and
//    term displacements are scalar), one column block at a time with two in flight.
//  * Nothing spills: a value reloaded from scratch in the output phase would make each 16-row
//    block of stores wait for the previous block's to complete.
//  * The unit vectors go out through LDS half 1, free between the last k-block and the next
//    tile's first copies into it: each wave stages 16 rows x its 64 columns at a time (eight
//    rounds per tile) and reads them back so that each non-temporal store instruction covers
//    whole 128-byte lines (four rows x 256 bytes): 16-byte pieces of 16 rows per instruction
//    wrote 1.5x the bytes to HBM, and ordinary stores left the next kernel's reads behind the
//    L2's write-backs.
//  * Products run with the weight fragment as the first operand, so each lane ends up holding
//    four consecutive columns of one row.
// Tile t is side t % 2 (0: W_in), rows (t / 2) * 128 onwards.
constexpr int kWideRows = 128;
constexpr int kWideWaves = 8;
constexpr int kWideNb = 4;      // 16-column blocks per wave
constexpr int kWideDkp = 16;    // 32-deep k-blocks
constexpr int kHalfChunks = 32; // 16-byte chunks per half row (256 bf16)
constexpr int kHalfStride = kHalfChunks * 16 + 16;  // bytes per half row in LDS (padded)
constexpr size_t kWideHalfBytes = (size_t)kWideRows * kHalfStride;
constexpr int kStageRows = 16;                  // output rows per wave per staging round
constexpr int kNonTemporal = 2;                 // cache-policy bits of a non-temporal store
constexpr int kStageStride = kWideNb * 16 + 4;  // floats per staged output row (padded)
static_assert((size_t)kWideWaves * kStageRows * kStageStride * sizeof(float) <= kWideHalfBytes,
              "the output staging fits in LDS half 1");

// B fragments of one piece through a buffer descriptor: one lane offset, the k-block and term
// displacements in the scalar offset, the column-block steps in the instruction offset
template <int NBP>
__device__ __forceinline__ void wide_bpiece(BFrag<NBP>& dst, __amdgpu_buffer_rsrc_t rs,
                                            uint32_t voff, uint32_t sbase, uint32_t slice, int kb) {
#pragma unroll
  for (int t = 0; t < 3; ++t) {
    const uint32_t so = sbase + (uint32_t)(kb * 3 + t) * slice;
#pragma unroll
    for (int j = 0; j < NBP; ++j)
      dst[j][t] = __builtin_bit_cast(
          u32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, voff + (uint32_t)j * 1024u, so, 0));
  }
}

// acc[mb][NBP g + j] += W-fragment x E-fragment over one k-block for column blocks NBP g ..
template <int NBP>
__device__ __forceinline__ void wide_mfma(f32x4 (&acc)[8][kWideNb], const BFrag<NBP>& b,
                                          const bf16x8 (&a)[8], int g) {
#pragma unroll
  for (int t = 0; t < 3; ++t)
#pragma unroll
    for (int mb = 0; mb < 8; ++mb)
#pragma unroll
      for (int j = 0; j < NBP; ++j)
        acc[mb][NBP * g + j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
            __builtin_bit_cast(bf16x8, b[j][t]), a[mb], acc[mb][NBP * g + j], 0, 0, 0);
}

__global__ __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(2, 2)))
void cand_vectors_wide_kernel(const int32_t* __restrict__ ids, const uint16_t* __restrict__ E,
                              const unsigned char* __restrict__ frags, int64_t M, int64_t V,
                              int d, int nbp, int64_t ntiles, float* __restrict__ in_vec,
                              float* __restrict__ out_vec) {
  constexpr int ROWS = kWideRows, NW = kWideWaves;
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  const int tid = threadIdx.x, lane = lane_id(),
            wave = (int)__builtin_amdgcn_readfirstlane((uint32_t)(tid / kWave));
  unsigned char* A = smem;                                                // [2][ROWS][32][16 B]
  float* ssbuf = reinterpret_cast<float*>(smem + 2 * kWideHalfBytes);    // [NW][ROWS]
  int32_t* rid = reinterpret_cast<int32_t*>(ssbuf + NW * ROWS);          // [3][ROWS]
  const size_t slice = (size_t)nbp * 1024;
  const int64_t step = gridDim.x;
  const __amdgpu_buffer_rsrc_t rsrc = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(E), (short)0, (int)(V * d * 2), 0x00020000);
  const uint32_t kOut = 0x80000000u;
  const int dchunks = d / 8;
  const __amdgpu_buffer_rsrc_t irs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<int32_t*>(ids), (short)0, (int)(M * (int64_t)sizeof(int32_t)), 0x00020000);
  const __amdgpu_buffer_rsrc_t frs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<unsigned char*>(frags), (short)0, (int)(2 * kWideDkp * 3 * slice), 0x00020000);  // 16-byte chunks per embedding row (d % 16 == 0)

  auto tile_id = [&](int64_t t) -> int32_t {
    int32_t v = -1;
    if (t < ntiles && tid < ROWS) {
      const int64_t row = (t >> 1) * ROWS + tid;
      if (row < M) {
        const int32_t id = ids[row];
        v = (id >= 0 && id < V) ? id : -1;
      }
    }
    return v;
  };
  // half h of row `row` of the tile whose ids are in rr: lanes 0..31, one 16-byte chunk each
  // (the row number passes through an empty asm so the compiler computes each copy's addresses
  // where the copy is issued instead of hoisting all of them out of the tile loop into registers)
  auto dma_half_id = [&](int32_t id, int h, int row) {
    __asm__ volatile("" : "+s"(row));
    if (lane < kHalfChunks) {
      const int c = h * kHalfChunks + lane;
      const uint32_t off = ((uint32_t)id < (uint32_t)V && c < dchunks)
                               ? (uint32_t)id * (uint32_t)(d * 2) + (uint32_t)c * 16u
                               : kOut;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          rsrc, (lds_ptr_t)(A + h * kWideHalfBytes + (size_t)row * kHalfStride), 16, off, 0, 0, 0);
    }
  };
  auto dma_half = [&](const int32_t* rr, int h, int row) {
    dma_half_id(__builtin_amdgcn_readfirstlane(rr[row]), h, row);
  };

  int64_t t = blockIdx.x;
  {
    const int32_t v0 = tile_id(t), v1 = tile_id(t + step);
    if (tid < ROWS) {
      rid[tid] = v0;
      rid[ROWS + tid] = v1;
    }
  }
  __syncthreads();
  // the first tile's first half; its second half arrives during its first k-blocks
  for (int r = wave; r < ROWS; r += NW) dma_half(rid, 0, r);
  __asm__ volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();

  for (int it = 0; t < ntiles; ++it, t += step) {
    // ids in LDS: slot it % 3 this tile's, (it + 1) % 3 the next tile's (both read just below)
    const int cur = it % 3, nxt = cur == 2 ? 0 : cur + 1, after = nxt == 2 ? 0 : nxt + 1;
    const bool has_next = t + step < ntiles;
    const int32_t* rc = rid + cur * ROWS;
    const int32_t* rn = rid + nxt * ROWS;
    const int side = (int)(t & 1);
    const uint32_t sbase = (uint32_t)(side * kWideDkp * 3) * (uint32_t)slice;
    const uint32_t voff = (uint32_t)(wave * kWideNb * 1024 + lane * 16);
    // ids of the rows this wave copies, lane j holding row wave + 8 j (j < 16): this tile's (for
    // its second half) and the next tile's (for its first half), read once so that a copy needs
    // no LDS read in the k-loop
    const int32_t idc = rc[(wave + NW * (lane & (ROWS / NW - 1))) & (ROWS - 1)];
    const int32_t idn = rn[(wave + NW * (lane & (ROWS / NW - 1))) & (ROWS - 1)];
    // the ids of the tile after the next are copied by the first two waves straight into slot
    // (it + 2) % 3 (read by no one during this tile), so no wave waits for them here; rows past
    // M read as id 0 (their outputs are dropped) and ids outside the vocabulary are caught where
    // a copy is issued. The copy has landed by the waits at this tile's end.
    if (wave < ROWS / kWave && t + 2 * step < ntiles) {
      const int64_t row = ((t + 2 * step) >> 1) * ROWS + wave * kWave + lane;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          irs, (lds_ptr_t)(rid + after * ROWS + wave * kWave), 4,
          row < M ? (uint32_t)row * 4u : kOut, 0, 0, 0);
    }

    f32x4 acc[8][kWideNb];
#pragma unroll
    for (int mb = 0; mb < 8; ++mb)
#pragma unroll
      for (int nb = 0; nb < kWideNb; ++nb) acc[mb][nb] = f32x4{0.f, 0.f, 0.f, 0.f};
    // the weight fragments of a k-block come in pieces of kPieceNb column blocks through
    // kBufs register buffers: while a piece is multiplied the next kBufs - 1 are in flight
    constexpr int kPieceNb = 1, kPieces = kWideNb / kPieceNb, kBufs = 3;
    constexpr int kTotalPieces = kWideDkp * kPieces;
    BFrag<kPieceNb> bq[kBufs];
    auto load_piece = [&](int p) {
      wide_bpiece<kPieceNb>(bq[p % kBufs], frs, voff + (uint32_t)((p % kPieces) * kPieceNb * 1024),
                            sbase, (uint32_t)slice, p / kPieces);
    };
#pragma unroll
    for (int p = 0; p < kBufs - 1; ++p) load_piece(p);
    const int arow = lane & 15, agrp = lane >> 4;
    // k-blocks kb0 .. kb0+7 from LDS half h. Two half-row copies per k-block go into the other
    // half: this tile's second half while the first is multiplied (that half was released at
    // the previous tile's end), the next tile's first half while the second is multiplied.
    auto kloop = [&](int kb0, int h) {
      const unsigned char* Ah = A + h * kWideHalfBytes;
#pragma unroll
      for (int kb = kb0; kb < kb0 + 8; ++kb) {
        // the two waves of a SIMD take turns by progress: a wave lowers its issue priority as it
        // moves through the k-blocks, so the one behind is served first and both reach the
        // barrier together
        if ((kb & 3) == 0) {
          if (kb == 0) __builtin_amdgcn_s_setprio(3);
          else if (kb == 4) __builtin_amdgcn_s_setprio(2);
          else if (kb == 8) __builtin_amdgcn_s_setprio(1);
          else __builtin_amdgcn_s_setprio(0);
        }
        __builtin_amdgcn_sched_barrier(0);
        constexpr int kCopies = ROWS / NW / 8;  // half-row copies per wave per k-block
        if (h == 0) {
#pragma unroll
          for (int i = 0; i < kCopies; ++i) {
            const int j = kCopies * (kb - kb0) + i;
            dma_half_id(__builtin_amdgcn_readlane(idc, j), 1, wave + NW * j);
          }
        } else if (has_next) {
#pragma unroll
          for (int i = 0; i < kCopies; ++i) {
            const int j = kCopies * (kb - kb0) + i;
            dma_half_id(__builtin_amdgcn_readlane(idn, j), 0, wave + NW * j);
          }
        }
        __builtin_amdgcn_sched_barrier(0);
        bf16x8 a[8];
        const unsigned char* Ak = Ah + arow * kHalfStride + ((kb & 7) * 4 + agrp) * 16;
#pragma unroll
        for (int mb = 0; mb < 8; ++mb)
          a[mb] = __builtin_bit_cast(
              bf16x8, *reinterpret_cast<const u32x4*>(Ak + mb * 16 * kHalfStride));
#pragma unroll
        for (int g = 0; g < kPieces; ++g) {
          const int p = kb * kPieces + g;
          if (p + kBufs - 1 < kTotalPieces) load_piece(p + kBufs - 1);
          __builtin_amdgcn_sched_barrier(0);
          wide_mfma<kPieceNb>(acc, bq[p % kBufs], a, g);
          __builtin_amdgcn_sched_barrier(0);
        }
      }
    };
    kloop(0, 0);
    // every wave is done with the first half, and the second half has landed: this wave's
    // copies, then everyone's
    __asm__ volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    kloop(8, 1);

    // this wave's 64-column part of every row's squared norm: lane l holds row 16 mb + l % 16,
    // columns 16 nb + 4 (l / 16) + i
#pragma unroll
    for (int mb = 0; mb < 8; ++mb) {
      float s = 0.f;
#pragma unroll
      for (int nb = 0; nb < kWideNb; ++nb)
#pragma unroll
        for (int i = 0; i < 4; ++i) s = fmaf(acc[mb][nb][i], acc[mb][nb][i], s);
      s += __shfl_xor(s, 16, kWave);
      s += __shfl_xor(s, 32, kWave);
      if (lane < 16) ssbuf[wave * ROWS + mb * 16 + lane] = s;
    }
    // the next tile's first half has landed and nobody reads this tile's second half any more
    __asm__ volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();

    float* out = side == 0 ? in_vec : out_vec;
    const int64_t row0 = (t >> 1) * ROWS;
    // the tile's output rows through a buffer descriptor bounded to the rows that exist, so a
    // store needs one 32-bit offset add and rows past M are dropped by the range check (the
    // 64-bit base moves with the tile, so only the tile's own 256 KB need 32-bit offsets)
    const int64_t out_bytes = (M - row0) * d * (int64_t)sizeof(float);
    const __amdgpu_buffer_rsrc_t orsrc = __builtin_amdgcn_make_buffer_rsrc(
        out + row0 * d, (short)0, (int)(out_bytes < 0x7fffffff ? out_bytes : 0x7fffffff),
        0x00020000);
    // the lane's row and column group, recomputed here (through an empty asm) rather than kept
    // in registers from the top of the kernel: a value reloaded from scratch between the stores
    // would make each 16-row block wait for the previous block's stores to complete
    int le = lane;
    __asm__ volatile("" : "+v"(le));
    const int er = le & 15, eg = le >> 4;
    // the output leaves through LDS half 1 (free until the next tile's copies into it begin):
    // each wave stages kStageRows rows x its 64 columns at a time, read back so that each 16
    // lanes write 256 contiguous bytes (whole lines) of one row with non-temporal stores
    float* stage = reinterpret_cast<float*>(A + kWideHalfBytes) + wave * kStageRows * kStageStride;
    const int col_w = wave * kWideNb * 16;
#pragma unroll
    for (int rnd = 0; rnd < ROWS / kStageRows; ++rnd) {
#pragma unroll
      for (int m2 = 0; m2 < kStageRows / 16; ++m2) {
        const int mb = rnd * (kStageRows / 16) + m2;
        const int rl = mb * 16 + er;
        float tot = 0.f;
#pragma unroll
        for (int w = 0; w < NW; ++w) tot += ssbuf[w * ROWS + rl];
        const float inv = tot > 0.f ? 1.0f / sqrtf(tot) : 0.f;
#pragma unroll
        for (int nb = 0; nb < kWideNb; ++nb)
          *reinterpret_cast<f32x4*>(stage + (m2 * 16 + er) * kStageStride + nb * 16 + eg * 4) =
              acc[mb][nb] * inv;
      }
      // lane: row 4 q + le / 16 of the round, columns col .. col + 3 (past d: outside the range)
      const int col = col_w + (le & 15) * 4;
      const uint32_t lane_off =
          col < d ? (uint32_t)(((le >> 4) * d + col) * (int)sizeof(float)) : 0x80000000u;
#pragma unroll
      for (int q = 0; q < kStageRows / 4; ++q) {
        const int sr = 4 * q + (le >> 4);
        const f32x4 v =
            *reinterpret_cast<const f32x4*>(stage + sr * kStageStride + (le & 15) * 4);
        const uint32_t row_off = (uint32_t)((rnd * kStageRows + 4 * q) * d * (int)sizeof(float));
        __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), orsrc,
                                               lane_off + row_off, 0, kNonTemporal);
      }
    }
    // every wave has read its staged rows back before the next tile's copies go into half 1
    __syncthreads();
  }
}

// Workgroups that run at once (one per compute unit), per device
int compute_units() {
  static int cached[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 0;
  if (cached[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
      return 0;
    cached[dev] = n;
  }
  return cached[dev];
}

constexpr int kF32Rows = 16;
constexpr int kF32Threads = 256;

__global__ __launch_bounds__(kF32Threads) void cand_vectors_f32_kernel(
    const int32_t* __restrict__ ids, const float* __restrict__ E, const float* __restrict__ Wf,
    int64_t M, int64_t V, int d, float* __restrict__ in_vec, float* __restrict__ out_vec) {
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  float* e = reinterpret_cast<float*>(smem);       // [16][d]
  float* part = e + kF32Rows * d;                  // [16][256]
  float* inv = part + kF32Rows * kF32Threads;      // [16]
  const int side = blockIdx.y;
  const int64_t r0 = blockIdx.x * (int64_t)kF32Rows;
  const int tid = threadIdx.x;
  for (int i = tid; i < kF32Rows * d; i += kF32Threads) {
    const int r = i / d, c = i % d;
    const int64_t row = r0 + r;
    const int32_t id = row < M ? ids[row] : -1;
    e[i] = (id >= 0 && id < V) ? E[(int64_t)id * d + c] : 0.f;  // outside [0, V): zero row
  }
  __syncthreads();
  const float* W = Wf + (size_t)side * d * d;
  float u[4][kF32Rows];
  float ss[kF32Rows];
#pragma unroll
  for (int r = 0; r < kF32Rows; ++r) ss[r] = 0.f;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int j = tid + q * kF32Threads;
#pragma unroll
    for (int r = 0; r < kF32Rows; ++r) u[q][r] = 0.f;
    if (j < d) {
      // unrolled so that several weight loads are in flight at once (d is a multiple of 16)
#pragma unroll 16
      for (int i = 0; i < d; ++i) {
        const float w = W[(int64_t)i * d + j];
#pragma unroll
        for (int r = 0; r < kF32Rows; ++r) u[q][r] = fmaf(e[r * d + i], w, u[q][r]);
      }
#pragma unroll
      for (int r = 0; r < kF32Rows; ++r) ss[r] = fmaf(u[q][r], u[q][r], ss[r]);
    }
  }
#pragma unroll
  for (int r = 0; r < kF32Rows; ++r) part[r * kF32Threads + tid] = ss[r];
  __syncthreads();
  if (tid < kF32Rows) {
    float t = 0.f;
    for (int i = 0; i < kF32Threads; ++i) t += part[tid * kF32Threads + i];
    inv[tid] = t > 0.f ? 1.0f / sqrtf(t) : 0.f;
  }
  __syncthreads();
  float* out = side == 0 ? in_vec : out_vec;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int j = tid + q * kF32Threads;
    if (j < d) {
#pragma unroll
      for (int r = 0; r < kF32Rows; ++r) {
        const int64_t row = r0 + r;
        if (row < M) out[row * d + j] = u[q][r] * inv[r];
      }
    }
  }
}

bool vec_d_ok(int d) { return d >= 16 && d <= 1024 && d % 16 == 0; }

}  // namespace
}  // namespace lilicorr

using namespace lilicorr;

extern "C" size_t lilicorr_packed_weight_bytes(int d) {
  if (!vec_d_ok(d)) return 0;
  return packed_bytes(d);
}

extern "C" lilicorr_status lilicorr_pack_weights(const float* W_in, const float* W_out, int d,
                                                 void* packed, hipStream_t stream) {
  if (!W_in || !W_out || !packed) return LILICORR_ERR_INVALID_ARG;
  if (!vec_d_ok(d)) return LILICORR_ERR_UNSUPPORTED;
  if (!aligned16(W_in) || !aligned16(W_out) || !aligned16(packed)) return LILICORR_ERR_ALIGNMENT;
  unsigned char* p = static_cast<unsigned char*>(packed);
  const VecGeom g = vec_geom(d);
  hipLaunchKernelGGL(pack_weights_kernel, dim3(1024), dim3(256), 0, stream, W_in, W_out, d, g.nbp,
                     g.dkp, reinterpret_cast<uint16_t*>(p),
                     reinterpret_cast<float*>(p + frag_bytes(d)));
  return launch_status();
}

extern "C" lilicorr_status lilicorr_candidate_vectors(const int32_t* ids, const void* E,
                                                      lilicorr_dtype e_dtype, int64_t V, int d,
                                                      const void* packed_w, int64_t N, int64_t B,
                                                      int K, float* in_vec, float* out_vec,
                                                      hipStream_t stream) {
  if (!ids || !E || !packed_w || !in_vec || !out_vec) return LILICORR_ERR_INVALID_ARG;
  if (e_dtype != LILICORR_F32 && e_dtype != LILICORR_BF16) return LILICORR_ERR_INVALID_ARG;
  if (N < 1 || B < 1 || K < 1 || V < 1) return LILICORR_ERR_INVALID_ARG;
  if (!vec_d_ok(d) || K > 64 || V >= ((int64_t)1 << 31)) return LILICORR_ERR_UNSUPPORTED;
  if (N > ((int64_t)1 << 40) / B) return LILICORR_ERR_UNSUPPORTED;
  const int64_t M = N * B * K;
  if (M > ((int64_t)1 << 40)) return LILICORR_ERR_UNSUPPORTED;
  if (!aligned16(ids) || !aligned16(E) || !aligned16(packed_w) || !aligned16(in_vec) ||
      !aligned16(out_vec))
    return LILICORR_ERR_ALIGNMENT;
  const unsigned char* p = static_cast<const unsigned char*>(packed_w);
  if (e_dtype == LILICORR_BF16) {
    const VecGeom g = vec_geom(d, M);
    const int64_t rows_wg = (int64_t)g.rm * 16;
    const int64_t nblk = (M + rows_wg - 1) / rows_wg;
    if (nblk > 0x7fffffffll) return LILICORR_ERR_UNSUPPORTED;
    const int ncu = compute_units();
    // at 448 < d <= 512, from one 128-row tile per compute unit: the wide persistent kernel (E
    // and the ids addressable by 32-bit buffer offsets)
    if (g.dkp == kWideDkp && g.nbp == kWideWaves * kWideNb && ncu > 0 &&
        2 * ((M + kWideRows - 1) / kWideRows) >= (int64_t)ncu &&
        V * d * 2 < ((int64_t)1 << 31) && M * 4 < ((int64_t)1 << 31)) {
      const int64_t wt = 2 * ((M + kWideRows - 1) / kWideRows);
      const int grid = (int)(wt < ncu ? wt : ncu);
      const size_t lds = 2 * kWideHalfBytes + (size_t)kWideWaves * kWideRows * sizeof(float) +
                         (size_t)3 * kWideRows * sizeof(int32_t);
      static const hipError_t attrw = hipFuncSetAttribute(
          reinterpret_cast<const void*>(cand_vectors_wide_kernel),
          hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
      (void)attrw;
      hipLaunchKernelGGL(cand_vectors_wide_kernel, dim3((unsigned)grid), dim3(kWideWaves * kWave),
                         lds, stream, ids, static_cast<const uint16_t*>(E), p, M, V, d, g.nbp, wt,
                         in_vec, out_vec);
      return launch_status();
    }
    const size_t lds = (size_t)rows_wg * (g.dkp * 32 + 8) * 2 +
                       (size_t)g.waves * rows_wg * sizeof(float) + (size_t)rows_wg * sizeof(int32_t);
    const dim3 grid((unsigned)nblk, 2), block(g.waves * kWave);
    const uint16_t* e16 = static_cast<const uint16_t*>(E);
    if (g.rm == 4) {
      static const hipError_t attr4 = hipFuncSetAttribute(
          reinterpret_cast<const void*>(cand_vectors_mfma_kernel<4, 512>),
          hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
      (void)attr4;
      hipLaunchKernelGGL((cand_vectors_mfma_kernel<4, 512>), grid, block, lds, stream, ids, e16, p,
                         M, V, d, g.nbp, g.dkp, in_vec, out_vec);
    } else {
      static const hipError_t attr2 = hipFuncSetAttribute(
          reinterpret_cast<const void*>(cand_vectors_mfma_kernel<2, 1024>),
          hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
      (void)attr2;
      hipLaunchKernelGGL((cand_vectors_mfma_kernel<2, 1024>), grid, block, lds, stream, ids, e16, p,
                         M, V, d, g.nbp, g.dkp, in_vec, out_vec);
    }
  } else {
    const int64_t nblk = (M + kF32Rows - 1) / kF32Rows;
    if (nblk > 0x7fffffffll) return LILICORR_ERR_UNSUPPORTED;
    const size_t lds = ((size_t)kF32Rows * d + kF32Rows * kF32Threads + kF32Rows) * sizeof(float);
    static const hipError_t attr_f32 = hipFuncSetAttribute(
        reinterpret_cast<const void*>(cand_vectors_f32_kernel),
        hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
    (void)attr_f32;
    hipLaunchKernelGGL(cand_vectors_f32_kernel, dim3((unsigned)nblk, 2), dim3(kF32Threads), lds,
                       stream, ids, static_cast<const float*>(E),
                       reinterpret_cast<const float*>(p + frag_bytes(d)), M, V, d, in_vec, out_vec);
  }
  return launch_status();
}
