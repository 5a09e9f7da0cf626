// Decode-path product for M <= 4 tokens (online phase of Appendix A, Eq. 2).
//
// Work mapping (one workgroup = one 64-row tile of T, 4 waves):
//  - lane i of every wave owns row 64*r + i, so the activations of a
//    container (128 weights) are the same for the whole wave and are read
//    with scalar loads into SGPRs;
//  - the 4 waves split the tile's 128-weight containers into 4 contiguous
//    ranges and combine their int32 partial sums through LDS at the end;
//  - a container is two contiguous wave-wide loads: 16-byte heads (1 KB)
//    and 4-byte tails (256 B) of the 64 rows' 160-bit code streams.
// Per code: one funnel shift + mask give code*4, one LDS read of the
// 32-entry decode table gives the int8x4 weights, one v_dot4 per token adds
// x . w into the int32 accumulator.  The decode table has one dword per
// code, so any 64 lookups are bank-conflict free.
#include <utility>

#include "sherry_internal.h"

namespace sherry {
namespace {

constexpr int kGemvThreads = 256;
constexpr int kPrefetch = 4;  // containers loaded per wave before decoding

// Byte offset (code*4) of code j of a 160-bit container held in d[0..4].
template <int j>
__device__ __forceinline__ uint32_t code_x4(const uint32_t (&d)[5]) {
  constexpr int bit = 5 * j, i = bit >> 5, off = bit & 31;
  if constexpr (off >= 2) {
    constexpr int hi = (i < 4) ? i + 1 : i;
    return __builtin_amdgcn_alignbit(d[hi], d[i], off - 2) & 0x7Cu;
  } else if constexpr (i > 0) {
    return __builtin_amdgcn_alignbit(d[i], d[i - 1], 30 + off) & 0x7Cu;
  } else {
    return (d[0] << 2) & 0x7Cu;
  }
}

// Codes are processed in groups of kGroup: the group's table offsets are
// computed first, then all its LDS reads are issued, then the dot products
// run, so kGroup reads are in flight per wave instead of one.
constexpr int kGroup = 16;

template <int j0, int... js>
__device__ __forceinline__ void group_offsets(const uint32_t (&d)[5], uint32_t* a4,
                                              std::integer_sequence<int, js...>) {
  ((a4[js] = code_x4<j0 + js>(d)), ...);
}

template <int M, bool kTail>
__device__ __forceinline__ void dot_codes(const uint32_t (&d)[5],
                                          const SHERRY_CONST int32_t* __restrict__ xw,
                                          int k_words_left, int kw,
                                          const uint32_t* lut, int32_t (&acc)[M]) {
#pragma unroll
  for (int g = 0; g < 32; g += kGroup) {
    int32_t xv[M][kGroup];
#pragma unroll
    for (int m = 0; m < M; ++m)
#pragma unroll
      for (int j = 0; j < kGroup; ++j) {
        if constexpr (kTail) xv[m][j] = (g + j < k_words_left) ? xw[m * kw + g + j] : 0;
        else xv[m][j] = xw[m * kw + g + j];
      }
    uint32_t a4[kGroup];
    if (g == 0) group_offsets<0>(d, a4, std::make_integer_sequence<int, kGroup>{});
    else group_offsets<kGroup>(d, a4, std::make_integer_sequence<int, kGroup>{});
    uint32_t wv[kGroup];
#pragma unroll
    for (int j = 0; j < kGroup; ++j)
      wv[j] = *reinterpret_cast<const uint32_t*>(reinterpret_cast<const char*>(lut) + a4[j]);
#pragma unroll
    for (int j = 0; j < kGroup; ++j)
#pragma unroll
      for (int m = 0; m < M; ++m)
        acc[m] = __builtin_amdgcn_sdot4(xv[m][j], static_cast<int32_t>(wv[j]), acc[m], false);
  }
}

template <int M>
__device__ __forceinline__ void gemv_tile(const uint8_t* w_, const int8_t* x_,
                                          const float* x_scale, float w_scale, float* y,
                                          int32_t* acc_out, int64_t n, int k, int r,
                                          const uint32_t* lut, int32_t* red) {
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int C = (k + kTileK - 1) / kTileK;
  const int c0 = (wave * C) >> 2, c1 = ((wave + 1) * C) >> 2;
  const SHERRY_GLOBAL uint8_t* tile = as_global(w_) + int64_t(r) * C * kUnitBytes;
  const SHERRY_CONST int32_t* xw0 = as_const(reinterpret_cast<const int32_t*>(x_));
  const int kw = k >> 2;

  int32_t acc[M];
#pragma unroll
  for (int m = 0; m < M; ++m) acc[m] = 0;

  for (int c = c0; c < c1; c += kPrefetch) {
    uint32_t d[kPrefetch][5];
#pragma unroll
    for (int u = 0; u < kPrefetch; ++u) {
      if (c + u < c1) {
        const SHERRY_GLOBAL uint8_t* unit = tile + int64_t(c + u) * kUnitBytes;
        const u32x4 h = *reinterpret_cast<const SHERRY_GLOBAL u32x4*>(unit + 16 * lane);
        d[u][0] = h.x;
        d[u][1] = h.y;
        d[u][2] = h.z;
        d[u][3] = h.w;
        d[u][4] = *reinterpret_cast<const SHERRY_GLOBAL uint32_t*>(unit + kHeadBytes + 4 * lane);
      }
    }
#pragma unroll
    for (int u = 0; u < kPrefetch; ++u) {
      if (c + u < c1) {
        const int kb = (c + u) * kTileK;
        const SHERRY_CONST int32_t* xw = xw0 + (kb >> 2);
        if (kb + kTileK <= k) {
          dot_codes<M, false>(d[u], xw, 32, kw, lut, acc);
        } else {
          dot_codes<M, true>(d[u], xw, (k - kb) >> 2, kw, lut, acc);
        }
      }
    }
  }

#pragma unroll
  for (int m = 0; m < M; ++m) red[(wave * M + m) * 64 + lane] = acc[m];
  __syncthreads();
  if (threadIdx.x < 64 * M) {
    const int m = threadIdx.x >> 6;
    const int i = threadIdx.x & 63;
    const int32_t a = red[(0 * M + m) * 64 + i] + red[(1 * M + m) * 64 + i] +
                      red[(2 * M + m) * 64 + i] + red[(3 * M + m) * 64 + i];
    const int64_t row = int64_t(r) * kTileRows + i;
    if (row < n) {
      const float s = as_const(x_scale)[m] * w_scale;
      as_global_mut(y)[m * n + row] = static_cast<float>(a) * s;
      if (acc_out) as_global_mut(acc_out)[m * n + row] = a;
    }
  }
}

__device__ __forceinline__ void fill_lut(uint32_t* lut) {
  if (threadIdx.x < 32) lut[threadIdx.x] = decode_word(threadIdx.x);
  __syncthreads();
}

template <int M>
__global__ __launch_bounds__(kGemvThreads) void gemv_kernel(
    const uint8_t* __restrict__ w, const int8_t* __restrict__ x,
    const float* __restrict__ x_scale, float w_scale, float* __restrict__ y,
    int32_t* __restrict__ acc, int64_t n, int64_t k) {
  __shared__ uint32_t lut[32];
  __shared__ int32_t red[4 * M * 64];
  fill_lut(lut);
  gemv_tile<M>(w, x, x_scale, w_scale, y, acc, n, static_cast<int>(k), blockIdx.x, lut, red);
}

__global__ __launch_bounds__(kGemvThreads) void gemv_batched_kernel(
    const sherry_gemv_desc* __restrict__ descs, int count) {
  __shared__ uint32_t lut[32];
  __shared__ int32_t red[4 * 64];
  fill_lut(lut);
  const int32_t tile = static_cast<int32_t>(blockIdx.x);
  int lo = 0, hi = count - 1;  // last descriptor with tile_begin <= tile
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (descs[mid].tile_begin <= tile) lo = mid;
    else hi = mid - 1;
  }
  const sherry_gemv_desc& d = descs[lo];
  gemv_tile<1>(d.w, d.x, d.x_scale, d.w_scale, d.y, d.acc, d.n, static_cast<int>(d.k),
               tile - d.tile_begin, lut, red);
}

}  // namespace

int launch_gemv_valu(const uint8_t* w, const int8_t* x, const float* x_scale, float w_scale,
                     float* y, int32_t* acc, int64_t m, int64_t n, int64_t k, hipStream_t s) {
  const dim3 grid(static_cast<unsigned>(ceil_div(n, kTileRows)));
  switch (m) {
    case 1:
      return launch(gemv_kernel<1>, grid, dim3(kGemvThreads), 0, s, w, x, x_scale,
                         w_scale, y, acc, n, k);
    case 2:
      return launch(gemv_kernel<2>, grid, dim3(kGemvThreads), 0, s, w, x, x_scale,
                         w_scale, y, acc, n, k);
    case 3:
      return launch(gemv_kernel<3>, grid, dim3(kGemvThreads), 0, s, w, x, x_scale,
                         w_scale, y, acc, n, k);
    case 4:
      return launch(gemv_kernel<4>, grid, dim3(kGemvThreads), 0, s, w, x, x_scale,
                         w_scale, y, acc, n, k);
    default:
      return SHERRY_E_SHAPE;
  }
}

int launch_gemv_batched(const sherry_gemv_desc* descs, int count, int64_t total_tiles,
                        hipStream_t s) {
  return launch(gemv_batched_kernel, dim3(static_cast<unsigned>(total_tiles)),
                     dim3(kGemvThreads), 0, s, descs, count);
}

}  // namespace sherry
