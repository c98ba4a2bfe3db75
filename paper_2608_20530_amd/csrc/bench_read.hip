// Measurement aid for bench.py, not part of the path: a plain streaming read of a device buffer
// with the same 16-byte, streaming-policy buffer loads as the logits pass, so the logits pass can
// be reported beside the read bandwidth this GPU reaches on the same bytes.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
constexpr int kThreads = 256;
constexpr int kUnroll = 8;

__global__ __launch_bounds__(kThreads) void stream_read_kernel(const u32x4* __restrict__ p,
                                                               int64_t n16,
                                                               uint32_t* __restrict__ sink) {
  // n16 * 16 bytes fit the descriptor's 32-bit range: the host splits larger buffers. Each
  // workgroup streams one contiguous segment, as the logits pass streams one row per workgroup
  // (measured well above a grid-strided sweep of the same bytes).
  const __amdgpu_buffer_rsrc_t rsrc = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<u32x4*>(p), (short)0, (int)(n16 * 16), 0x00020000);
  const int64_t per = (n16 + gridDim.x - 1) / gridDim.x;
  const int64_t begin = (int64_t)blockIdx.x * per;
  const int64_t end = begin + per < n16 ? begin + per : n16;
  uint32_t acc = 0;
  for (int64_t base = begin + threadIdx.x; base < end; base += (int64_t)kThreads * kUnroll) {
    u32x4 v[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int64_t i = base + u * kThreads;
      // past the segment: an offset outside the descriptor reads zeros without memory traffic
      const uint32_t off = i < end ? (uint32_t)(i * 16) : 0xFFFFFFF0u;
      v[u] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rsrc, off, 0, 3));
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
  }
  sink[(int64_t)blockIdx.x * kThreads + threadIdx.x] = acc;
}

}  // namespace

// Reads `bytes` (a multiple of 16, 16-byte aligned) from p; sink holds grid * 256 words.
// Returns 0 on success, -1 on bad arguments, -5 if the launch failed.
extern "C" int bench_stream_read(const void* p, size_t bytes, uint32_t* sink, int grid,
                                 hipStream_t stream) {
  if (!p || !sink || grid < 1 || bytes % 16 != 0 || (reinterpret_cast<uintptr_t>(p) & 15u))
    return -1;
  const size_t kPiece = (size_t)1 << 30;  // per launch, inside the descriptor's range
  for (size_t off = 0; off < bytes; off += kPiece) {
    const size_t n = bytes - off < kPiece ? bytes - off : kPiece;
    hipLaunchKernelGGL(stream_read_kernel, dim3(grid), dim3(kThreads), 0, stream,
                       reinterpret_cast<const u32x4*>(static_cast<const char*>(p) + off),
                       (int64_t)(n / 16), sink);
  }
  return hipGetLastError() == hipSuccess ? 0 : -5;
}
