// Sparse-AbsMean ternarization and packing on the GPU (Eq. 4 and Eq. 5):
// fp32 weights in, the packed 5-bit tiled layout and one alpha per output
// channel out, with the same bytes as sherry_pack applied to the ternary
// matrix of Eq. 4.
//
// Work mapping.  A workgroup owns RW rows (64, 32 or 16) of one 64-row tile
// and all of their units; lane l of a wave is row l % RW and unit slot l / RW,
// so a lane turns one row of one unit (128 weights) into its 16-byte head
// and 4-byte tail directly.  Each lane reads its 128 values as 32 16-byte
// loads (one block of 4 per load).  Fewer rows per workgroup give small-N
// matrices more workgroups.  The kept magnitudes are summed in fp64 per
// lane and the partial sums of each row are added in a fixed order.
#include "sherry_internal.h"

namespace sherry {
namespace {

constexpr int kTpWaves = 8;
constexpr int kTpThreads = 64 * kTpWaves;

// Code of one block (Eq. 4): the smallest |w| is dropped (ties to the lowest
// position); the other three keep their sign, +1 for a kept zero.  Adds the
// kept magnitudes to kept.
__device__ __forceinline__ uint32_t tp_block(const float4 v, double& kept) {
  const float w[4] = {v.x, v.y, v.z, v.w};
  const float a[4] = {fabsf(v.x), fabsf(v.y), fabsf(v.z), fabsf(v.w)};
  int z = 0;
#pragma unroll
  for (int p = 1; p < 4; ++p) z = (a[p] < a[z]) ? p : z;
  uint32_t neg = 0;  // sign bit of the i-th kept weight, ascending position
  int i = 0;
#pragma unroll
  for (int p = 0; p < 4; ++p) {
    if (p == z) continue;
    neg |= (w[p] < 0.0f ? 1u : 0u) << i;
    kept += static_cast<double>(a[p]);
    ++i;
  }
  return static_cast<uint32_t>(z) | (neg << 2);
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
__device__ __forceinline__ void tp_unit(const float* row_w, bool in, int64_t b0, int64_t nb,
                                        uint32_t (&d)[5], double& kept,
                                        std::integer_sequence<int, js...>) {
  (
      [&] {
        const int64_t b = b0 + js;
        uint32_t code = 0;  // padding rows and blocks hold code 0
        if (in && b < nb) {
          const float4 v = *reinterpret_cast<const float4*>(as_global(row_w + 4 * b));
          code = tp_block(v, kept);
        }
        tp_put<js>(d, code);
      }(),
      ...);
}

template <int RW>
__global__ __launch_bounds__(kTpThreads) void ternarize_pack_kernel(
    const float* __restrict__ w, int64_t n, int64_t k, uint8_t* __restrict__ out,
    float* __restrict__ alpha) {
  constexpr int SLOTS = 64 / RW;  // units in flight per wave
  __shared__ double red[kTpWaves * 64];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int64_t r = blockIdx.x / SLOTS;           // tile
  const int ri = (blockIdx.x % SLOTS) * RW + lane % RW;  // row within the tile
  const int64_t row = r * kTileRows + ri;
  const int64_t C = (k + kTileK - 1) / kTileK, nb = k / 4;
  const bool in = row < n;
  const float* row_w = w + (in ? row : 0) * k;
  double kept = 0.0;
  for (int64_t c = wave * SLOTS + lane / RW; c < C; c += kTpWaves * SLOTS) {
    uint32_t d[5] = {0, 0, 0, 0, 0};
    tp_unit(row_w, in, c * 32, nb, d, kept, std::make_integer_sequence<int, 32>{});
    uint8_t* unit = out + (r * C + c) * kUnitBytes;
    *reinterpret_cast<uint4*>(as_global_mut(unit + 16 * ri)) = make_uint4(d[0], d[1], d[2], d[3]);
    *reinterpret_cast<uint32_t*>(as_global_mut(unit + kHeadBytes + 4 * ri)) = d[4];
  }
  red[wave * 64 + lane] = kept;
  __syncthreads();
  if (threadIdx.x < RW) {
    const int64_t arow = r * kTileRows + (blockIdx.x % SLOTS) * RW + threadIdx.x;
    if (arow < n && alpha) {
      double s = 0.0;
      for (int q = 0; q < kTpWaves * SLOTS; ++q)  // wave-major, then slot
        s += red[(q / SLOTS) * 64 + (q % SLOTS) * RW + threadIdx.x];
      // Eq. 5: mean |W| over the row's kept weights (three per block)
      as_global_mut(alpha)[arow] = static_cast<float>(s / static_cast<double>(3 * nb));
    }
  }
}

}  // namespace

int launch_ternarize_pack(const float* w, int64_t n, int64_t k, uint8_t* out, float* alpha,
                          hipStream_t s) {
  const int64_t R = ceil_div(n, kTileRows);
  const dim3 block(kTpThreads);
  // rows per workgroup: whole tiles when there are enough of them
  if (R >= 256)
    return launch(ternarize_pack_kernel<64>, dim3(static_cast<unsigned>(R)), block, 0, s, w, n,
                  k, out, alpha);
  if (R >= 128)
    return launch(ternarize_pack_kernel<32>, dim3(static_cast<unsigned>(2 * R)), block, 0, s, w,
                  n, k, out, alpha);
  return launch(ternarize_pack_kernel<16>, dim3(static_cast<unsigned>(4 * R)), block, 0, s, w, n,
                k, out, alpha);
}

}  // namespace sherry
