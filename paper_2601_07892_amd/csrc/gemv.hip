// Decode-path product for M <= 4 tokens (online phase of Appendix A, Eq. 2).
//
// Work mapping.  A workgroup is 4 waves; lane i of a wave owns row 64*r + i
// of one 64-row tile r, so the activations of a container (128 weights) are
// the same for the whole wave and live in SGPRs (scalar loads).  Each tile's
// containers are split among S = gemv_split(C) waves (1, 2 or 4, so that a
// wave streams about 16 containers); a workgroup covers 4/S tiles and its
// waves combine their int32 partial sums through LDS.
//
// Streaming.  A container is two contiguous wave-wide loads: the 64 rows'
// 16-byte heads (1 KB) and 4-byte tails (256 B).  Each wave double-buffers
// two register sets of kSet containers: one set is in flight while the
// other is decoded.
//
// Decode.  Per code: a funnel shift and mask (or one SDWA mask) give code*4,
// one LDS read of the 32-entry table gives the int8x4 weights, one v_dot4 per
// token accumulates x . w in int32.  The table holds one dword per code, so
// any 64 lookups are free of bank conflicts; codes are processed in groups
// so 8 or 16 table reads are in flight.
#include <utility>

#include "sherry_internal.h"

namespace sherry {
namespace {

constexpr int kGemvThreads = 256;
constexpr int kSet = 4;  // containers per register set (two sets per wave)

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

template <int j0, int... js>
__device__ __forceinline__ void group_offsets(const uint32_t (&d)[5], uint32_t* a4,
                                              std::integer_sequence<int, js...>) {
  ((a4[js] = code_x4<j0 + js>(d)), ...);
}

// Codes decoded per batch of table reads: 16 for one token; 8 when several
// tokens' activation words must sit in SGPRs at once.
template <int M>
constexpr int group_size() { return M == 1 ? 16 : 8; }

// Decodes codes [g, g + G) of a container in d[0..4] and accumulates the dot
// products with the activation words at xw (M tokens, row stride kw words,
// wave-uniform: scalar loads into SGPRs).  Words at or beyond words_left read
// as zero (last, partial container).
template <int M, bool kTail, int g = 0>
__device__ __forceinline__ void dot_container(const uint32_t (&d)[5],
                                              const SHERRY_CONST int32_t* xw, int kw,
                                              int words_left, const uint32_t* lut,
                                              int32_t (&acc)[M]) {
  constexpr int G = group_size<M>();
  if constexpr (g < 32) {
    // keep each group's loads, table reads and dot products together: the
    // scheduler would otherwise hoist every group's loads and run out of
    // scalar registers
    __builtin_amdgcn_sched_barrier(0);
    int32_t xv[M][G];
#pragma unroll
    for (int m = 0; m < M; ++m)
#pragma unroll
      for (int j = 0; j < G; ++j) {
        if constexpr (kTail) {
          // branch-free: read an in-bounds word, then zero it past K
          const int idx = (g + j < words_left) ? g + j : words_left - 1;
          const int32_t v = xw[m * kw + idx];
          xv[m][j] = (g + j < words_left) ? v : 0;
        } else {
          xv[m][j] = xw[m * kw + g + j];
        }
      }
    uint32_t a4[G];
    group_offsets<g>(d, a4, std::make_integer_sequence<int, G>{});
    uint32_t wv[G];
#pragma unroll
    for (int j = 0; j < G; ++j)
      wv[j] = *reinterpret_cast<const uint32_t*>(reinterpret_cast<const char*>(lut) + a4[j]);
#pragma unroll
    for (int j = 0; j < G; ++j)
#pragma unroll
      for (int m = 0; m < M; ++m)
        acc[m] = __builtin_amdgcn_sdot4(xv[m][j], static_cast<int32_t>(wv[j]), acc[m], false);
    dot_container<M, kTail, g + G>(d, xw, kw, words_left, lut, acc);
  }
}

// Container c of a tile through a buffer resource spanning exactly that
// tile's containers (reads outside it return zero, never fault): 16-byte
// head at lane*16, 4-byte tail at 1024 + lane*4, container offset in SGPRs.
__device__ __forceinline__ void load_container(uint32_t (&d)[5], __amdgpu_buffer_rsrc_t r,
                                               int c, int lane) {
  const u32x4 h = __builtin_amdgcn_raw_buffer_load_b128(r, 16 * lane, c * kUnitBytes, 0);
  d[0] = h.x;
  d[1] = h.y;
  d[2] = h.z;
  d[3] = h.w;
  d[4] = __builtin_amdgcn_raw_buffer_load_b32(r, kHeadBytes + 4 * lane, c * kUnitBytes, 0);
}

template <int P>
__device__ __forceinline__ void load_set(uint32_t (&d)[P][5], __amdgpu_buffer_rsrc_t r, int c,
                                         int lane) {
#pragma unroll
  for (int u = 0; u < P; ++u) load_container(d[u], r, c + u, lane);
}

template <int M>
__device__ __forceinline__ void dot_any(const uint32_t (&d)[5], int cc,
                                        const SHERRY_CONST int32_t* xw0, int k,
                                        const uint32_t* lut, int32_t (&acc)[M]) {
  const int kb = cc * kTileK;
  if (kb + kTileK <= k) dot_container<M, false>(d, xw0 + (kb >> 2), k >> 2, 32, lut, acc);
  else dot_container<M, true>(d, xw0 + (kb >> 2), k >> 2, (k - kb) >> 2, lut, acc);
}

template <int M, int P>
__device__ __forceinline__ void dot_set(const uint32_t (&d)[P][5], int c,
                                        const SHERRY_CONST int32_t* xw0, int kw,
                                        const uint32_t* lut, int32_t (&acc)[M]) {
#pragma unroll
  for (int u = 0; u < P; ++u)
    dot_container<M, false>(d[u], xw0 + (c + u) * (kTileK / 4), kw, 32, lut, acc);
}

// Streams containers [c0, c1) of one tile with two register sets of kSet
// containers: set B is loaded while set A is decoded and the reverse, so
// kSet containers are always in flight.  Sets only cover full containers
// [c0, cf): cf excludes a partial last container at the end of K.  Every
// set load is issued only after checking it lies in [c0, cf); at the top of
// the loop the outstanding loads are always exactly set A's, so the compiler
// waits on exact counts.  What is left (fewer than kSet containers, and the
// partial one) is drained one container at a time.
template <int M>
__device__ __forceinline__ void stream_tile(__amdgpu_buffer_rsrc_t tile, int c0, int c1,
                                            const SHERRY_CONST int32_t* xw0, int k,
                                            const uint32_t* lut, int32_t (&acc)[M]) {
  const int lane = threadIdx.x & 63;
  const int kw = k >> 2;
  const int cf = (c1 * kTileK > k) ? c1 - 1 : c1;
  uint32_t a[kSet][5], b[kSet][5];
  int c = c0;
  if (c + kSet <= cf) {
    load_set<kSet>(a, tile, c, lane);
    while (true) {
      // set A holds [c, c + kSet), inside [c0, cf)
      if (c + 2 * kSet <= cf) {
        load_set<kSet>(b, tile, c + kSet, lane);
        dot_set<M, kSet>(a, c, xw0, kw, lut, acc);
        if (c + 3 * kSet <= cf) {
          load_set<kSet>(a, tile, c + 2 * kSet, lane);
          dot_set<M, kSet>(b, c + kSet, xw0, kw, lut, acc);
          c += 2 * kSet;
          continue;
        }
        dot_set<M, kSet>(b, c + kSet, xw0, kw, lut, acc);
        c += 2 * kSet;
        break;
      }
      dot_set<M, kSet>(a, c, xw0, kw, lut, acc);
      c += kSet;
      break;
    }
  }
  for (; c < c1; ++c) {
    uint32_t d[5];
    load_container(d, tile, c, lane);
    dot_any<M>(d, c, xw0, k, lut, acc);
  }
}

// One workgroup of a product: block g of a problem whose tiles are split
// over S waves each.
template <int M>
__device__ __forceinline__ void gemv_block(const uint8_t* w_, const int8_t* x_,
                                           const float* x_scale, float w_scale, float* y,
                                           int32_t* acc_out, int64_t n, int k, int g, int S,
                                           const uint32_t* lut, int32_t* red) {
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int C = (k + kTileK - 1) / kTileK;
  const int R = static_cast<int>((n + kTileRows - 1) / kTileRows);
  const int tpb = 4 / S;           // tiles per block
  const int lt = wave / S;         // tile of this wave inside the block
  const int part = wave - lt * S;  // part of the tile's containers
  const int r = g * tpb + lt;

  int32_t acc[M];
#pragma unroll
  for (int m = 0; m < M; ++m) acc[m] = 0;
  if (r < R) {
    const int c0 = (part * C) / S, c1 = ((part + 1) * C) / S;
    const __amdgpu_buffer_rsrc_t tile = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint8_t*>(w_) + int64_t(r) * C * kUnitBytes, 0, C * kUnitBytes,
        kBufferWord3);
    stream_tile<M>(tile, c0, c1, as_const(reinterpret_cast<const int32_t*>(x_)), k, lut, acc);
  }

#pragma unroll
  for (int m = 0; m < M; ++m) red[(wave * M + m) * 64 + lane] = acc[m];
  __syncthreads();
  // thread t -> (tile lt2, token m, row i); the S waves of a tile are adjacent
  for (int t = threadIdx.x; t < tpb * M * 64; t += kGemvThreads) {
    const int i = t & 63;
    const int m = (t >> 6) % M;
    const int lt2 = (t >> 6) / M;
    const int r2 = g * tpb + lt2;
    const int64_t row = int64_t(r2) * kTileRows + i;
    if (r2 >= R || row >= n) continue;
    int32_t a = 0;
    for (int p = 0; p < S; ++p) a += red[((lt2 * S + p) * M + m) * 64 + i];
    const float s = as_const(x_scale)[m] * w_scale;
    as_global_mut(y)[m * n + row] = static_cast<float>(a) * s;
    if (acc_out) as_global_mut(acc_out)[m * n + row] = a;
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
    int32_t* __restrict__ acc, int64_t n, int64_t k, int split) {
  __shared__ uint32_t lut[32];
  __shared__ int32_t red[4 * M * 64];
  fill_lut(lut);
  gemv_block<M>(w, x, x_scale, w_scale, y, acc, n, static_cast<int>(k), blockIdx.x, split, lut,
                red);
}

__global__ __launch_bounds__(kGemvThreads) void gemv_batched_kernel(
    const sherry_gemv_desc* __restrict__ descs, int count) {
  __shared__ uint32_t lut[32];
  __shared__ int32_t red[4 * 64];
  fill_lut(lut);
  const int32_t blk = static_cast<int32_t>(blockIdx.x);
  int lo = 0, hi = count - 1;  // last descriptor with block_begin <= blk
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (descs[mid].block_begin <= blk) lo = mid;
    else hi = mid - 1;
  }
  const sherry_gemv_desc& d = descs[lo];
  const int k = static_cast<int>(d.k);
  const int S = gemv_split(static_cast<int>((k + kTileK - 1) / kTileK));
  gemv_block<1>(d.w, d.x, d.x_scale, d.w_scale, d.y, d.acc, d.n, k, blk - d.block_begin, S,
                lut, red);
}

}  // namespace

int launch_gemv_valu(const uint8_t* w, const int8_t* x, const float* x_scale, float w_scale,
                     float* y, int32_t* acc, int64_t m, int64_t n, int64_t k, hipStream_t s) {
  const int64_t R = ceil_div(n, kTileRows);
  const int C = static_cast<int>(ceil_div(k, kTileK));
  // a lone launch has only this product to fill the GPU: split every tile
  // over 4 waves unless there are plenty of tiles
  const int S = (R * gemv_split(C) >= 2048) ? gemv_split(C) : 4;
  const dim3 grid(static_cast<unsigned>(ceil_div(R * S, 4)));
  const dim3 block(kGemvThreads);
  switch (m) {
    case 1: return launch(gemv_kernel<1>, grid, block, 0, s, w, x, x_scale, w_scale, y, acc, n, k, S);
    case 2: return launch(gemv_kernel<2>, grid, block, 0, s, w, x, x_scale, w_scale, y, acc, n, k, S);
    case 3: return launch(gemv_kernel<3>, grid, block, 0, s, w, x, x_scale, w_scale, y, acc, n, k, S);
    case 4: return launch(gemv_kernel<4>, grid, block, 0, s, w, x, x_scale, w_scale, y, acc, n, k, S);
    default: return SHERRY_E_SHAPE;
  }
}

int launch_gemv_batched(const sherry_gemv_desc* descs, int count, int64_t total_blocks,
                        hipStream_t s) {
  return launch(gemv_batched_kernel, dim3(static_cast<unsigned>(total_blocks)),
                dim3(kGemvThreads), 0, s, descs, count);
}

}  // namespace sherry
