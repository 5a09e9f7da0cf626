// One-token product through activation lookup tables: the table direction of
// the paper's CPU engine (Sec. 3.1 and Appendix A) mapped onto the GPU, as a
// measured comparison point for the weight-table kernel of gemv.hip.
//
// Per block of 4 activations the workgroup builds, in LDS, the 16 dot
// products of the block with the canonical patterns: the codes whose third
// sign bit s2 is clear.  Flipping all three signs mirrors a pattern,
// decode(c ^ 0b11100) = -decode(c), so a code's contribution is the entry of
// its 4-bit index, (c & 15) ^ (s2 ? 12 : 0), negated when s2 is set: one
// sign bit and four index bits, as the paper splits its 5-bit code.
//
// Work mapping as in gemv.hip: lane i of a wave owns row i of a 64-row tile,
// a tile's containers are split over S waves whose int32 partial sums meet
// in LDS.  Entries are int16 (|entry| <= 3 * 128), 32 bytes per block, so
// the table of the longest row (SHERRY_ALUT_MAX_K values) takes 64 KB.
#include "sherry_internal.h"

namespace sherry {
namespace {

constexpr int kAlutWaves = 8;
constexpr int kAlutThreads = 64 * kAlutWaves;

// Contribution of code j of a container (its 16 table rows at tb).
template <int j>
__device__ __forceinline__ int32_t alut_term(const uint32_t (&d)[5], const int16_t* tb) {
  const uint32_t c = code_x4<j>(d) >> 2;  // the 5-bit code
  const uint32_t s2 = c >> 4;
  const uint32_t idx = (c & 15u) ^ (s2 * 12u);
  const int32_t v = tb[j * 16 + idx];
  return s2 ? -v : v;
}

template <int... js>
__device__ __forceinline__ int32_t alut_container(const uint32_t (&d)[5], const int16_t* tb,
                                                  std::integer_sequence<int, js...>) {
  return (alut_term<js>(d, tb) + ...);
}

__global__ __launch_bounds__(kAlutThreads) void gemv_alut_kernel(
    const uint8_t* __restrict__ w, const int8_t* __restrict__ x,
    const float* __restrict__ x_scale, WScale ws, float* __restrict__ y,
    int32_t* __restrict__ acc_out, int64_t n, int k, int S) {
  __shared__ __attribute__((aligned(16))) int16_t tab[SHERRY_ALUT_MAX_K / 4 * 16];
  __shared__ int32_t red[kAlutWaves * 64];
  const int C = (k + kTileK - 1) / kTileK;
  const int nb = k >> 2;
  // the tables of every block of the row (blocks past k, up to whole
  // containers, hold zeros: their codes are padding)
  for (int e = threadIdx.x; e < C * 32 * 16; e += kAlutThreads) {
    const int b = e >> 4;
    int32_t v = 0;
    if (b < nb) {
      const int32_t x4 = as_global(reinterpret_cast<const int32_t*>(x))[b];
      v = __builtin_amdgcn_sdot4(x4, static_cast<int32_t>(decode_word(e & 15)), 0, false);
    }
    tab[e] = static_cast<int16_t>(v);
  }
  __syncthreads();

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int R = static_cast<int>((n + kTileRows - 1) / kTileRows);
  const int tpb = kAlutWaves / S;
  const int lt = wave / S, part = wave - lt * S;
  const int r = blockIdx.x * tpb + lt;
  const int c0 = (r < R) ? (part * C) / S : 0, c1 = (r < R) ? ((part + 1) * C) / S : 0;
  const UnitRun rs{w + (int64_t(r < R ? r : 0) * C + c0) * kUnitBytes, c1 - c0};
  int32_t acc = 0;
  uint32_t cur[5], nxt[5];
  load_unit(cur, rs, 0, lane);  // past the range: zeros, no memory access
  for (int i = 0; i < c1 - c0; ++i) {
    load_unit(nxt, rs, i + 1, lane);
    acc += alut_container(cur, tab + (c0 + i) * 32 * 16, std::make_integer_sequence<int, 32>{});
#pragma unroll
    for (int q = 0; q < 5; ++q) cur[q] = nxt[q];
  }

  red[wave * 64 + lane] = acc;
  __syncthreads();
  if (static_cast<int>(threadIdx.x) < tpb * 64) {
    const int lt2 = threadIdx.x >> 6, i = threadIdx.x & 63;
    const int r2 = blockIdx.x * tpb + lt2;
    const int64_t row = int64_t(r2) * kTileRows + i;
    if (r2 < R && row < n) {
      int32_t a = 0;
      for (int p = 0; p < S; ++p) a += red[(lt2 * S + p) * 64 + i];
      as_global_mut(y)[row] = static_cast<float>(a) * (as_global(x_scale)[0] * ws.at(row));
      if (acc_out) as_global_mut(acc_out)[row] = a;
    }
  }
}

}  // namespace

int launch_gemv_alut(const uint8_t* w, const int8_t* x, const float* x_scale, WScale ws,
                     float* y, int32_t* acc, int64_t n, int64_t k, hipStream_t s) {
  if (k > SHERRY_ALUT_MAX_K) return SHERRY_E_SHAPE;
  const int64_t R = ceil_div(n, kTileRows);
  const int C = static_cast<int>(ceil_div(k, kTileK));
  const int S = (R * gemv_split(C) >= 4096) ? gemv_split(C) : kAlutWaves;
  return launch(gemv_alut_kernel, dim3(static_cast<unsigned>(ceil_div(R * S, kAlutWaves))),
                dim3(kAlutThreads), 0, s, w, x, x_scale, ws, y, acc, n, static_cast<int>(k), S);
}

}  // namespace sherry
