// Streaming-read probe: the practical HBM read ceiling next to the 8 TB/s
// specification.  Each workgroup reads a contiguous slice with 128-bit loads
// and writes one XOR checksum word (so the loads cannot be elided).
#include "sherry_internal.h"

namespace sherry {
namespace {

constexpr int kThreads = 256;
constexpr int64_t kSliceBytes = 256 * 1024;  // per workgroup

__global__ __launch_bounds__(kThreads) void stream_read_kernel(const uint4* __restrict__ src,
                                                               int64_t n16,
                                                               uint32_t* __restrict__ sink) {
  __shared__ uint32_t part[kThreads / 64];
  const int64_t per = kSliceBytes / 16;
  const int64_t b = int64_t(blockIdx.x) * per;
  const int64_t e = (b + per < n16) ? b + per : n16;
  uint32_t h = 0;
  int64_t i = b + threadIdx.x;
  for (; i + 3 * kThreads < e; i += 4 * kThreads) {
    const uint4 a = src[i], c = src[i + kThreads], d = src[i + 2 * kThreads],
                f = src[i + 3 * kThreads];
    h ^= a.x ^ a.y ^ a.z ^ a.w ^ c.x ^ c.y ^ c.z ^ c.w ^ d.x ^ d.y ^ d.z ^ d.w ^ f.x ^ f.y ^
         f.z ^ f.w;
  }
  for (; i < e; i += kThreads) {
    const uint4 a = src[i];
    h ^= a.x ^ a.y ^ a.z ^ a.w;
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
                     0, s, static_cast<const uint4*>(src), static_cast<int64_t>(bytes / 16),
                     sink);
}

}  // namespace sherry
