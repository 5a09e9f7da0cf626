// Sparse-AbsMean ternarization and packing on the GPU (Eq. 4 and Eq. 5):
// fp32 weights in, the packed 5-bit tiled layout and one alpha per output
// channel out, with the same bytes as sherry_pack applied to the ternary
// matrix of Eq. 4.
//
// Work mapping.  A workgroup owns ROWS rows (16, 8 or 4) of one 64-row tile
// and every unit of them.  Its 32 * ROWS threads read the rows' weights one
// unit at a time, 32 consecutive lanes per row, each lane one block of 4
// (16 bytes): every wave load covers whole 512-byte row segments.  A lane
// turns its block into a code (Eq. 4) and adds the kept magnitudes to its
// fp64 partial sum.  The codes of 8 units go through LDS, and each unit row's
// 32 codes are then packed by one lane into its 16-byte head and 4-byte tail,
// while the next 8 units' loads are in flight.
// Rows past n, blocks past k and units past the padded row read as zeros
// (their offsets fall outside the range of the wave's buffer resource) and so
// become code 0, the padding code.  The alpha of a row (Eq. 5) adds its 32
// lanes' partial sums in a fixed order.
#include "sherry_internal.h"

namespace sherry {
namespace {

constexpr int kTpRound = 8;  // units in flight per round

// Code of one block (Eq. 4): the smallest |w| is dropped (ties to the lowest
// position); the other three keep their sign, +1 for a kept zero.  Adds the
// kept magnitudes to kept, in ascending position (the dropped one adds +0,
// which leaves the fp64 sum unchanged).  Branch-free: the sign bits of the
// four weights are gathered and the dropped position's bit is cut out.
__device__ __forceinline__ uint32_t tp_block(const float4 v, double& kept) {
  const float a0 = fabsf(v.x), a1 = fabsf(v.y), a2 = fabsf(v.z), a3 = fabsf(v.w);
  uint32_t z = 0;
  float lo = a0;
  if (a1 < lo) { z = 1; lo = a1; }
  if (a2 < lo) { z = 2; lo = a2; }
  if (a3 < lo) z = 3;
  const uint32_t s = (v.x < 0.0f ? 1u : 0u) | (v.y < 0.0f ? 2u : 0u) | (v.z < 0.0f ? 4u : 0u) |
                     (v.w < 0.0f ? 8u : 0u);
  const uint32_t neg = (s & ((1u << z) - 1u)) | ((s >> (z + 1u)) << z);
  kept += static_cast<double>(z == 0 ? 0.0f : a0);
  kept += static_cast<double>(z == 1 ? 0.0f : a1);
  kept += static_cast<double>(z == 2 ? 0.0f : a2);
  kept += static_cast<double>(z == 3 ? 0.0f : a3);
  return z | (neg << 2);
}

// Code j of a unit row sits at bits [5j, 5j + 5) of the 160-bit row
// (head words 0-3, tail word 4).
template <int j>
__device__ __forceinline__ void tp_put(uint32_t (&d)[5], uint32_t code) {
  constexpr int b = 5 * j, wd = b / 32, off = b % 32;
  d[wd] |= code << off;
  if constexpr (off > 27) d[wd + 1] |= code >> (32 - off);
}

template <int... js>
__device__ __forceinline__ void tp_pack(const uint8_t* codes, uint32_t (&d)[5],
                                        std::integer_sequence<int, js...>) {
  (tp_put<js>(d, codes[js]), ...);
}

template <int ROWS>
__global__ __launch_bounds__(32 * ROWS) void ternarize_pack_kernel(
    const float* __restrict__ w, int64_t n, int64_t k, uint8_t* __restrict__ out,
    float* __restrict__ alpha) {
  constexpr int THREADS = 32 * ROWS, WAVES = THREADS / 64;
  constexpr int QUARTERS = kTileRows / ROWS;  // workgroups per tile
  __shared__ __attribute__((aligned(16))) uint8_t codes[kTpRound][ROWS][32];
  __shared__ double part[ROWS][32];
  const int tid = threadIdx.x;
  const int rl = tid >> 5, j = tid & 31;  // row of the workgroup, block of the unit
  const int64_t tile = blockIdx.x / QUARTERS;
  const int r0 = (blockIdx.x % QUARTERS) * ROWS;  // first row within the tile
  const int64_t row = tile * kTileRows + r0 + rl;
  const int64_t C = (k + kTileK - 1) / kTileK, nb = k / 4;
  // one buffer resource per wave (it must be wave-uniform): the wave's two
  // rows, rows past n left out of its range; a lane's block past the end of
  // its row gets an offset past the range, so both read as zeros (k % 4 == 0,
  // so no block straddles two rows)
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int64_t wrow0 = tile * kTileRows + r0 + 2 * wave;  // rows rl & ~1 and rl | 1
  const int64_t wrows = n - wrow0 < 0 ? 0 : (n - wrow0 < 2 ? n - wrow0 : 2);
  const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<float*>(w) + (wrows > 0 ? wrow0 : 0) * k, 0, static_cast<int>(wrows * k * 4),
      kBufferWord3);
  const int rowoff = static_cast<int>((rl & 1) * k * 4);
  constexpr int kPastRange = 0x7ffffff0;
  double kept = 0.0;
  float4 v[kTpRound];
  auto load_round = [&](int64_t c0) {
#pragma unroll
    for (int u = 0; u < kTpRound; ++u) {
      const int64_t blk = (c0 + u) * 32 + j;
      const int off = blk < nb ? rowoff + static_cast<int>(blk * 16) : kPastRange;
      const u32x4 raw = __builtin_amdgcn_raw_buffer_load_b128(rs, off, 0, kLoadStream);
      v[u] = make_float4(__uint_as_float(raw.x), __uint_as_float(raw.y), __uint_as_float(raw.z),
                         __uint_as_float(raw.w));
    }
  };
  load_round(0);
  for (int64_t c0 = 0; c0 < C; c0 += kTpRound) {
#pragma unroll
    for (int u = 0; u < kTpRound; ++u) codes[u][rl][j] = static_cast<uint8_t>(tp_block(v[u], kept));
    // the next round's loads fly while this round is packed
    if (c0 + kTpRound < C) load_round(c0 + kTpRound);
    __syncthreads();
    // unit c0 + u, row lane: one lane per unit row packs its 32 codes
    const int lane = tid & 63;
    for (int u = wave; u < kTpRound; u += WAVES) {
      if (lane < ROWS && c0 + u < C) {
        uint32_t d[5] = {0, 0, 0, 0, 0};
        tp_pack(codes[u][lane], d, std::make_integer_sequence<int, 32>{});
        uint8_t* unit = out + (tile * C + c0 + u) * kUnitBytes;
        const int ri = r0 + lane;
        *reinterpret_cast<uint4*>(as_global_mut(unit + 16 * ri)) = make_uint4(d[0], d[1], d[2], d[3]);
        *reinterpret_cast<uint32_t*>(as_global_mut(unit + kHeadBytes + 4 * ri)) = d[4];
      }
    }
    __syncthreads();  // the next round rewrites codes
  }
  part[rl][j] = kept;
  __syncthreads();
  if (tid < ROWS) {
    const int64_t arow = tile * kTileRows + r0 + tid;
    if (arow < n && alpha) {
      double sum = 0.0;
      for (int q = 0; q < 32; ++q) sum += part[tid][q];  // ascending block position
      // Eq. 5: mean |W| over the row's kept weights (three per block)
      as_global_mut(alpha)[arow] = static_cast<float>(sum / static_cast<double>(3 * nb));
    }
  }
}

}  // namespace

int launch_ternarize_pack(const float* w, int64_t n, int64_t k, uint8_t* out, float* alpha,
                          hipStream_t s) {
  const int64_t R = ceil_div(n, kTileRows);
  // rows per workgroup: fewer for matrices with few tiles, so that there are
  // enough workgroups to spread over the GPU
  if (R >= 64)
    return launch(ternarize_pack_kernel<16>, dim3(static_cast<unsigned>(4 * R)), dim3(512), 0, s,
                  w, n, k, out, alpha);
  if (R >= 16)
    return launch(ternarize_pack_kernel<8>, dim3(static_cast<unsigned>(8 * R)), dim3(256), 0, s,
                  w, n, k, out, alpha);
  return launch(ternarize_pack_kernel<4>, dim3(static_cast<unsigned>(16 * R)), dim3(128), 0, s, w,
                n, k, out, alpha);
}

}  // namespace sherry
