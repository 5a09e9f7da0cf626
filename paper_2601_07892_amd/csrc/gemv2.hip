// Reference M = 1 product on the 2-bit layout (the "2-bit strategy" of
// Sec. 2.3, one ternary weight per 2 bits).  It exists only to compare bytes
// moved against the 1.25-bit layout on the same machine, so it mirrors the
// 5-bit kernel's mapping: one workgroup per 64-row tile, lane = row, 4 waves
// split the 64-weight units along K, activations in SGPRs, int32 partials
// combined through LDS.  Decode of 16 weights per dword: a 256-entry LDS
// table maps 4 two-bit values (one byte) to an int8x4 word.
#include "sherry_internal.h"

namespace sherry {
namespace {

constexpr int kThreads = 256;

__device__ __forceinline__ uint32_t decode_byte2(uint32_t b) {
  uint32_t word = 0;
  for (int p = 0; p < 4; ++p) {
    const uint32_t v = (b >> (2 * p)) & 3u;  // w + 1
    const uint32_t byte = (v == 0) ? 0xFFu : ((v == 2) ? 0x01u : 0x00u);
    word |= byte << (8 * p);
  }
  return word;
}

__global__ __launch_bounds__(kThreads) void gemv2_kernel(
    const uint8_t* __restrict__ w, const int8_t* __restrict__ x,
    const float* __restrict__ x_scale, float w_scale, float* __restrict__ y,
    int32_t* __restrict__ acc_out, int64_t n, int64_t k) {
  __shared__ uint32_t lut[256];
  __shared__ int32_t red[4 * 64];
  lut[threadIdx.x] = decode_byte2(threadIdx.x);
  __syncthreads();

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int64_t r = blockIdx.x;
  const int64_t C = (k + kTileK2 - 1) / kTileK2;
  const int64_t c0 = (wave * C) >> 2, c1 = ((wave + 1) * C) >> 2;
  const uint8_t* tile = w + r * C * kUnit2Bytes;
  const int32_t* xw0 = reinterpret_cast<const int32_t*>(x);
  int32_t acc = 0;
  for (int64_t c = c0; c < c1; ++c) {
    const uint4 h = *reinterpret_cast<const uint4*>(tile + c * kUnit2Bytes + 16 * lane);
    const uint32_t d[4] = {h.x, h.y, h.z, h.w};
    const int64_t kb = c * kTileK2;
    const int32_t* xw = xw0 + (kb >> 2);
    const int64_t left = (k - kb) >> 2;  // valid x words in this unit
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const uint32_t byte = (d[j >> 2] >> (8 * (j & 3))) & 0xFFu;
      const int32_t wv = static_cast<int32_t>(lut[byte]);
      const int32_t xv = (j < left) ? xw[j] : 0;
      acc = __builtin_amdgcn_sdot4(xv, wv, acc, false);
    }
  }
  red[wave * 64 + lane] = acc;
  __syncthreads();
  if (threadIdx.x < 64) {
    const int i = threadIdx.x;
    const int32_t a = red[i] + red[64 + i] + red[128 + i] + red[192 + i];
    const int64_t row = r * kTileRows + i;
    if (row < n) {
      y[row] = static_cast<float>(a) * (x_scale[0] * w_scale);
      if (acc_out) acc_out[row] = a;
    }
  }
}

}  // namespace

int launch_gemv2(const uint8_t* w2, const int8_t* x, const float* x_scale, float w_scale,
                 float* y, int32_t* acc, int64_t n, int64_t k, hipStream_t s) {
  return launch(gemv2_kernel, dim3(static_cast<unsigned>(ceil_div(n, kTileRows))),
                     dim3(kThreads), 0, s, w2, x, x_scale, w_scale, y, acc, n, k);
}

}  // namespace sherry
