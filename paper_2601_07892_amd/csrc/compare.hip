// M = 1 products on the two comparison layouts of Sec. 2.3: the "2-bit
// strategy" (one ternary weight per 2 bits) and the "1.67-bit strategy"
// (three ternary weights per 5-bit code, 27 of 32 codes used).  They exist to
// measure, on the same machine, what the 1.25-bit 3:4 layout saves in bytes
// and time, so they are built like its int8 GEMV: lane i of a wave owns row i
// of a 64-row tile, a tile's units are split among S waves of an 8-wave
// workgroup, each wave streams its units through a register ring with
// non-temporal buffer loads, the activations are wave-uniform words in SGPRs,
// v_dot4 accumulates in int32, and the S partial sums meet in LDS.
//
// 2-bit layout: unit = 64 rows x 64 weights, one 16-byte load per lane.  Byte
// p of the lane's word w holds the fields of weights 16w + p, 16w + 4 + p,
// 16w + 8 + p and 16w + 12 + p at bits 0, 2, 4 and 6, so one shift and one
// mask leave the values w + 1 of four consecutive weights in the four bytes
// of a register, ready for v_dot4 against one activation word.  v_dot4 then
// sums x . (w + 1); each wave subtracts the sum of its activations once.
//
// 1.67-bit layout: unit = 64 rows x 96 weights, stored like a 5-bit unit
// (16-byte head + 4-byte tail per lane, code j at stream bits [5j, 5j + 5)).
// Per code: the same funnel shift and mask as the 5-bit layout, one read of a
// 32-entry LDS table (int8 weights t0, t1, t2 and a zero byte), one v_dot4.
// The three activations of code j start at byte 3j: the scalar unit cuts them
// out of the SGPR words (a funnel shift of two words), the table's zero byte
// hides the fourth.  This is the 3-way alignment cost of the layout.
#include <utility>

#include "sherry_internal.h"

namespace sherry {
namespace {

constexpr int kWaves = 8;
constexpr int kThreads = 64 * kWaves;
constexpr int kRing = 3;

struct TwoBit {
  static constexpr int kK = kTileK2;        // weights per unit row
  static constexpr int kBytes = kUnit2Bytes;
  static constexpr int kTarget = 20;        // units per wave (1 KB units)
  static constexpr bool kSumCorrection = true;
  __device__ static void load(uint32_t (&d)[5], const UnitRun& run, int c, int lane) {
    const u32x4 h =
        __builtin_amdgcn_raw_buffer_load_b128(run.unit<kBytes>(c), 16 * lane, 0, kLoadStream);
    d[0] = h.x;
    d[1] = h.y;
    d[2] = h.z;
    d[3] = h.w;
    d[4] = 0;
  }
  // xw: the unit's 16 activation words (wave-uniform)
  __device__ static int32_t dot(const uint32_t (&d)[5], const int32_t (&xw)[kK / 4],
                                const uint32_t*, int32_t acc) {
#pragma unroll
    for (int w = 0; w < 4; ++w)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const uint32_t u = (d[w] >> (2 * j)) & 0x03030303u;
        acc = __builtin_amdgcn_sdot4(xw[4 * w + j], static_cast<int32_t>(u), acc, false);
      }
    return acc;
  }
};

struct Triple {
  static constexpr int kK = kTileK3;
  static constexpr int kBytes = kUnitBytes;
  static constexpr int kTarget = 16;
  static constexpr bool kSumCorrection = false;
  __device__ static void load(uint32_t (&d)[5], const UnitRun& run, int c, int lane) {
    load_unit(d, run, c, lane);
  }
  // Activation bytes 3j .. 3j + 3 of the unit (byte 3 meets the table's zero).
  template <int j>
  __device__ static int32_t act3(const int32_t (&xw)[kK / 4]) {
    constexpr int b = 3 * j, q = b >> 2, s = 8 * (b & 3);
    if constexpr (s == 0) {
      return xw[q];
    } else if constexpr (s == 8) {
      return static_cast<int32_t>(static_cast<uint32_t>(xw[q]) >> 8);
    } else {
      return static_cast<int32_t>((static_cast<uint32_t>(xw[q]) >> s) |
                                  (static_cast<uint32_t>(xw[q + 1]) << (32 - s)));
    }
  }
  // codes [g, g + 16): 16 table reads in flight, then 16 v_dot4
  template <int g, int... js>
  __device__ static void dot16(const uint32_t (&d)[5], const int32_t (&xw)[kK / 4],
                               const uint32_t* lut, int32_t& acc,
                               std::integer_sequence<int, js...>) {
    uint32_t wv[16];
    ((wv[js] = *reinterpret_cast<const uint32_t*>(reinterpret_cast<const char*>(lut) +
                                                  code_x4<g + js>(d))), ...);
    ((acc = __builtin_amdgcn_sdot4(act3<g + js>(xw), static_cast<int32_t>(wv[js]), acc, false)),
     ...);
  }
  template <int g>
  __device__ static void dot_group(const uint32_t (&d)[5], const int32_t (&xw)[kK / 4],
                                   const uint32_t* lut, int32_t& acc) {
    if constexpr (g < 32) {
      __builtin_amdgcn_sched_barrier(0);
      dot16<g>(d, xw, lut, acc, std::make_integer_sequence<int, 16>{});
      dot_group<g + 16>(d, xw, lut, acc);
    }
  }
  __device__ static int32_t dot(const uint32_t (&d)[5], const int32_t (&xw)[kK / 4],
                                const uint32_t* lut, int32_t acc) {
    dot_group<0>(d, xw, lut, acc);
    return acc;
  }
};

// Weights of a 1.67-bit code as an int8x4 word: byte q = base-3 digit q minus
// one (q = 0, 1, 2), byte 3 zero; the five unused codes decode to zero.
__device__ __forceinline__ uint32_t decode3_word(uint32_t code) {
  if (code > 26) return 0;
  uint32_t word = 0;
  for (int q = 0; q < 3; ++q, code /= 3) word |= ((code % 3 + 0xFFu) & 0xFFu) << (8 * q);
  return word;
}

// The unit's activation words, wave-uniform (scalar loads).  In a unit that
// crosses k, words at or past k read the last word of the row (in bounds) and
// are zeroed.
template <class L>
__device__ __forceinline__ void unit_words(const SHERRY_CONST int32_t* x, int k, int c,
                                           int32_t (&xw)[L::kK / 4]) {
  const int base = c * (L::kK / 4), left = (k >> 2) - base;
  if (left >= L::kK / 4) {
#pragma unroll
    for (int i = 0; i < L::kK / 4; ++i) xw[i] = x[base + i];
  } else {
#pragma unroll
    for (int i = 0; i < L::kK / 4; ++i) {
      const int32_t v = x[base + (i < left ? i : left - 1)];
      xw[i] = i < left ? v : 0;
    }
  }
}

__device__ __forceinline__ int32_t wave_sum_i32(int32_t v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

// One workgroup: block g of a product whose tiles are split over S waves.
template <class L>
__device__ __forceinline__ void cmp_block(const uint8_t* w, const int8_t* x_, const float* x_scale,
                                          float w_scale, float* y, int32_t* acc_out, int64_t n,
                                          int k, int g, int S, const uint32_t* lut, int32_t* red) {
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int C = (k + L::kK - 1) / L::kK;
  const int R = static_cast<int>((n + kTileRows - 1) / kTileRows);
  const int tpb = kWaves / S;
  const int lt = wave / S;
  const int part = wave - lt * S;
  const int r = g * tpb + lt;
  const int c0 = (r < R) ? (part * C) / S : 0, c1 = (r < R) ? ((part + 1) * C) / S : 0;
  const UnitRun range{w + (int64_t(r < R ? r : 0) * C + c0) * L::kBytes, c1 - c0};
  const SHERRY_CONST int32_t* x = as_const(reinterpret_cast<const int32_t*>(x_));
  // 2-bit: sum of the activations of this wave's K range, read by the whole
  // wave before the stream starts
  int32_t xsum = 0;
  if constexpr (L::kSumCorrection) {
    const int w0 = c0 * (L::kK / 4);
    const int w1 = min(c1 * (L::kK / 4), k >> 2);
    for (int i = w0 + lane; i < w1; i += 64)
      xsum = __builtin_amdgcn_sdot4(as_global(reinterpret_cast<const int32_t*>(x_))[i],
                                    0x01010101, xsum, false);
  }
  uint32_t ring[kRing][5];
#pragma unroll
  for (int u = 0; u < kRing; ++u) {
    L::load(ring[u], range, u, lane);
    __builtin_amdgcn_sched_barrier(0);
  }
  int32_t acc = 0;
  const int nu = c1 - c0;
  for (int i = 0; i < nu; i += kRing) {
#pragma unroll
    for (int u = 0; u < kRing; ++u) {
      if (i + u < nu) {
        int32_t xw[L::kK / 4];
        unit_words<L>(x, k, c0 + i + u, xw);
        acc = L::dot(ring[u], xw, lut, acc);
      }
      __builtin_amdgcn_sched_barrier(0);
      L::load(ring[u], range, i + u + kRing, lane);
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  if constexpr (L::kSumCorrection) acc -= wave_sum_i32(xsum);
  red[wave * 64 + lane] = acc;
  __syncthreads();
  for (int t = threadIdx.x; t < tpb * 64; t += kThreads) {
    const int i = t & 63, lt2 = t >> 6, r2 = g * tpb + lt2;
    const int64_t row = int64_t(r2) * kTileRows + i;
    if (r2 >= R || row >= n) continue;
    int32_t a = 0;
    for (int p = 0; p < S; ++p) a += red[(lt2 * S + p) * 64 + i];
    as_global_mut(y)[row] = static_cast<float>(a) * (as_const(x_scale)[0] * w_scale);
    if (acc_out) as_global_mut(acc_out)[row] = a;
  }
}

template <class L>
__device__ __forceinline__ void fill_table(uint32_t* lut) {
  if constexpr (!L::kSumCorrection) {
    if (threadIdx.x < 32) lut[threadIdx.x] = decode3_word(threadIdx.x);
    __syncthreads();
  }
}

template <class L>
__global__ __launch_bounds__(kThreads) void cmp_kernel(const uint8_t* __restrict__ w,
                                                       const int8_t* __restrict__ x,
                                                       const float* __restrict__ x_scale,
                                                       float w_scale, float* __restrict__ y,
                                                       int32_t* __restrict__ acc, int64_t n,
                                                       int k, int split) {
  __shared__ uint32_t lut[32];
  __shared__ int32_t red[kWaves * 64];
  fill_table<L>(lut);
  cmp_block<L>(w, x, x_scale, w_scale, y, acc, n, k, blockIdx.x, split, lut, red);
}

template <class L>
__global__ __launch_bounds__(kThreads) void cmp_batched_kernel(
    const sherry_gemv_desc* __restrict__ descs, int count) {
  __shared__ uint32_t lut[32];
  __shared__ int32_t red[kWaves * 64];
  fill_table<L>(lut);
  const int32_t blk = static_cast<int32_t>(blockIdx.x);
  // last descriptor with block_begin <= blk (a prefix: block_begin increases)
  const int lane = threadIdx.x & 63;
  int lo = 0;
  for (int base = 0; base < count; base += 64) {
    const int i = base + lane;
    const bool ok = i < count && as_global(descs)[i].block_begin <= blk;
    const int len = __popcll(__ballot(ok));
    lo = base + len - 1;
    if (len < 64) break;
  }
  lo = __builtin_amdgcn_readfirstlane(lo);
  const sherry_gemv_desc& d = descs[lo];
  const int k = static_cast<int>(d.k);
  const int S = gemv_split((k + L::kK - 1) / L::kK, L::kTarget);
  cmp_block<L>(d.w, d.x, d.x_scale, d.w_scale, d.y, d.acc, d.n, k, blk - d.block_begin, S, lut,
               red);
}

template <class L>
int64_t blocks_of(int64_t n, int64_t k) {
  const int S = gemv_split(static_cast<int>(ceil_div(k, L::kK)), L::kTarget);
  return ceil_div(ceil_div(n, kTileRows) * S, kWaves);
}

template <class L>
int launch_one(const uint8_t* w, const int8_t* x, const float* x_scale, float w_scale, float* y,
               int32_t* acc, int64_t n, int64_t k, hipStream_t s) {
  const int S = gemv_split(static_cast<int>(ceil_div(k, L::kK)), L::kTarget);
  return launch(cmp_kernel<L>, dim3(static_cast<unsigned>(blocks_of<L>(n, k))), dim3(kThreads),
                0, s, w, x, x_scale, w_scale, y, acc, n, static_cast<int>(k), S);
}

}  // namespace

int64_t cmp_blocks(int layout, int64_t n, int64_t k) {
  return layout == 2 ? blocks_of<TwoBit>(n, k) : blocks_of<Triple>(n, k);
}

int launch_gemv2(const uint8_t* w2, const int8_t* x, const float* x_scale, float w_scale,
                 float* y, int32_t* acc, int64_t n, int64_t k, hipStream_t s) {
  return launch_one<TwoBit>(w2, x, x_scale, w_scale, y, acc, n, k, s);
}

int launch_gemv3(const uint8_t* w3, const int8_t* x, const float* x_scale, float w_scale,
                 float* y, int32_t* acc, int64_t n, int64_t k, hipStream_t s) {
  return launch_one<Triple>(w3, x, x_scale, w_scale, y, acc, n, k, s);
}

int launch_cmp_batched(int layout, const sherry_gemv_desc* descs, int count,
                       int64_t total_blocks, hipStream_t s) {
  if (layout == 2)
    return launch(cmp_batched_kernel<TwoBit>, dim3(static_cast<unsigned>(total_blocks)),
                  dim3(kThreads), 0, s, descs, count);
  return launch(cmp_batched_kernel<Triple>, dim3(static_cast<unsigned>(total_blocks)),
                dim3(kThreads), 0, s, descs, count);
}

}  // namespace sherry
