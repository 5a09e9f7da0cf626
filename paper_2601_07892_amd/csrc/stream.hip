// Streaming-read probe: the practical HBM read ceiling next to the 8 TB/s
// specification, read the way the products read their packed weights: raw
// 128-bit buffer loads with the non-temporal hint.  Each workgroup reads a
// contiguous slice and writes one XOR checksum word (so the loads cannot be
// elided).
#include "sherry_internal.h"

namespace sherry {
namespace {

constexpr int kThreads = 256;
// 32 KB per workgroup: at the decode step's 155 MB per launch, 256 KB slices
// left too few workgroups in flight (25.8 us against 24.2 us); at 2 GiB the
// two read alike (7.0 TB/s)
constexpr int64_t kSliceBytes = 32 * 1024;  // per workgroup

__global__ __launch_bounds__(kThreads) void stream_read_kernel(const uint8_t* __restrict__ src,
                                                               int64_t bytes,
                                                               uint32_t* __restrict__ sink) {
  __shared__ uint32_t part[kThreads / 64];
  const int64_t b = int64_t(blockIdx.x) * kSliceBytes;
  const int64_t len = (b + kSliceBytes < bytes) ? kSliceBytes : bytes - b;
  // the resource spans exactly this slice: loads past it return zero
  const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(src) + b, 0, static_cast<int>(len), kBufferWord3);
  uint32_t h = 0;
  const int v = 16 * static_cast<int>(threadIdx.x);
  for (int off = 0; off < len; off += 4 * 16 * kThreads) {
    const u32x4 a = __builtin_amdgcn_raw_buffer_load_b128(r, v, off, kLoadStream);
    const u32x4 c = __builtin_amdgcn_raw_buffer_load_b128(r, v, off + 16 * kThreads, kLoadStream);
    const u32x4 d = __builtin_amdgcn_raw_buffer_load_b128(r, v, off + 32 * kThreads, kLoadStream);
    const u32x4 f = __builtin_amdgcn_raw_buffer_load_b128(r, v, off + 48 * kThreads, kLoadStream);
    h ^= a.x ^ a.y ^ a.z ^ a.w ^ c.x ^ c.y ^ c.z ^ c.w ^ d.x ^ d.y ^ d.z ^ d.w ^ f.x ^ f.y ^
         f.z ^ f.w;
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) h ^= __shfl_xor(h, off, 64);
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = h;
  __syncthreads();
  if (threadIdx.x == 0) sink[blockIdx.x] = part[0] ^ part[1] ^ part[2] ^ part[3];
}

}  // namespace

int64_t stream_read_groups(size_t bytes) {
  return static_cast<int64_t>((bytes + kSliceBytes - 1) / kSliceBytes);
}

int launch_stream_read(const void* src, size_t bytes, uint32_t* sink, hipStream_t s) {
  const int64_t groups = stream_read_groups(bytes);
  return launch(stream_read_kernel, dim3(static_cast<unsigned>(groups)), dim3(kThreads),
                     0, s, static_cast<const uint8_t*>(src), static_cast<int64_t>(bytes), sink);
}

}  // namespace sherry
