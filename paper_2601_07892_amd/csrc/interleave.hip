// Lane-interleaved units on the device: rewrites tiled units (as the host
// packer or sherry_ternarize_pack writes them) in the lane-interleaved
// layout that the matrix-core products read (defined in sherry.h).
#include "sherry_internal.h"

namespace sherry {
namespace {

// One wave per unit: the unit is read into LDS, then lane l gathers its 32
// codes (row 16g + t, block 16p + 4b + c for code 4(2g + p) + c, l = 16b + t)
// from the tiled containers and writes its own container.
__global__ __launch_bounds__(64) void interleave_kernel(const uint8_t* __restrict__ tiled,
                                                        uint8_t* __restrict__ il) {
  __shared__ uint32_t u32[kUnitBytes / 4];
  const int lane = threadIdx.x;
  const size_t base = static_cast<size_t>(blockIdx.x) * kUnitBytes;
  const uint32_t* src = reinterpret_cast<const uint32_t*>(tiled + base);
  for (int i = lane; i < kUnitBytes / 4; i += 64) u32[i] = src[i];
  __syncthreads();
  const int b = lane >> 4, t = lane & 15;
  uint32_t out[5] = {0u, 0u, 0u, 0u, 0u};
  for (int j = 0; j < 32; ++j) {
    const int g = j >> 3, p = (j >> 2) & 1, c = j & 3;
    const int row = 16 * g + t, block = 16 * p + 4 * b + c;
    // stream bit 5*block of row's container: dwords 0-3 are the head at
    // 16*row, dword 4 the tail at 1024 + 4*row
    const int sp = 5 * block, w = sp >> 5, s = sp & 31;
    auto word = [&](int q) { return q < 4 ? u32[4 * row + q] : u32[kHeadBytes / 4 + row]; };
    const uint64_t pair = static_cast<uint64_t>(word(w)) |
                          (w + 1 < 5 ? static_cast<uint64_t>(word(w + 1)) << 32 : 0ull);
    const uint32_t code = static_cast<uint32_t>(pair >> s) & 31u;
    const int dp = 5 * j, dw = dp >> 5, ds = dp & 31;
    out[dw] |= code << ds;
    if (ds > 27 && dw + 1 < 5) out[dw + 1] |= code >> (32 - ds);
  }
  uint32_t* dst = reinterpret_cast<uint32_t*>(il + base);
  for (int q = 0; q < 4; ++q) dst[4 * lane + q] = out[q];
  dst[kHeadBytes / 4 + lane] = out[4];
}

}  // namespace
}  // namespace sherry

using namespace sherry;

extern "C" int sherry_interleave(const uint8_t* tiled, uint8_t* il, int64_t n, int64_t k,
                                 void* stream) {
  if (!tiled || !il) return SHERRY_E_INVALID;
  if (sherry_packed_bytes(n, k) == 0) return SHERRY_E_SHAPE;
  if (tiled == il) return SHERRY_E_INVALID;
  if ((reinterpret_cast<uintptr_t>(tiled) & 15) || (reinterpret_cast<uintptr_t>(il) & 15))
    return SHERRY_E_ALIGN;
  const int64_t units = ceil_div(n, kTileRows) * ceil_div(k, kTileK);
  if (units > INT32_MAX) return SHERRY_E_SHAPE;
  return launch(interleave_kernel, dim3(static_cast<unsigned>(units)), dim3(64), 0,
                static_cast<hipStream_t>(stream), tiled, il);
}
