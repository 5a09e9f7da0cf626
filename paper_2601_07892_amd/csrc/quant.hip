// Per-token int8 activation quantization on the device.
//
// The paper keeps activations in BF16 (weights-only setting, Limitations) but
// its engine accumulates in integers (Appendix A, online phase).  The integer
// inputs are produced here: s = absmax/127, q = clamp(rint(x/s), -127, 127).
// One workgroup per token row.  Rows up to 16384 values are read once into
// registers; longer rows are read twice (absmax, then quantize).
#include "sherry_internal.h"

namespace sherry {
namespace {

constexpr int kQuantThreads = 256;

__device__ __forceinline__ float block_max(float amax, float* part) {
  amax = wave_max_f32(amax);
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = amax;
  __syncthreads();
  return fmaxf(fmaxf(part[0], part[1]), fmaxf(part[2], part[3]));
}

// Rows of up to NV*1024 values: the row is read once into registers (NV
// float4 per thread), reduced, and quantized from registers.
template <int NV>
__global__ __launch_bounds__(kQuantThreads) void quantize_rows_reg(
    const float* __restrict__ x, int64_t k, int8_t* __restrict__ q,
    float* __restrict__ x_scale) {
  __shared__ float part[kQuantThreads / 64];
  const int64_t row = blockIdx.x;
  const float4* xr = reinterpret_cast<const float4*>(x + row * k);
  uint32_t* qr = reinterpret_cast<uint32_t*>(q + row * k);
  const int k4 = static_cast<int>(k >> 2);
  float4 v[NV];
  float amax = 0.0f;
#pragma unroll
  for (int e = 0; e < NV; ++e) {
    const int i = threadIdx.x + e * kQuantThreads;
    v[e] = (i < k4) ? xr[i] : make_float4(0.f, 0.f, 0.f, 0.f);
    amax = fmaxf(amax, fmaxf(fmaxf(fabsf(v[e].x), fabsf(v[e].y)),
                             fmaxf(fabsf(v[e].z), fabsf(v[e].w))));
  }
  amax = block_max(amax, part);
  const float s = amax / 127.0f;
  const float rs = 1.0f / s;
#pragma unroll
  for (int e = 0; e < NV; ++e) {
    const int i = threadIdx.x + e * kQuantThreads;
    if (i < k4) qr[i] = (amax == 0.0f) ? 0u : quant4(v[e], s, rs);
  }
  if (threadIdx.x == 0) x_scale[row] = (amax == 0.0f) ? 0.0f : s;
}

// Any row length: two passes over the row (the second from cache).
__global__ __launch_bounds__(kQuantThreads) void quantize_rows(
    const float* __restrict__ x, int64_t k, int8_t* __restrict__ q,
    float* __restrict__ x_scale) {
  __shared__ float part[kQuantThreads / 64];
  const int64_t row = blockIdx.x;
  const float4* xr = reinterpret_cast<const float4*>(x + row * k);
  uint32_t* qr = reinterpret_cast<uint32_t*>(q + row * k);
  const int64_t k4 = k >> 2;

  float amax = 0.0f;
  for (int64_t i = threadIdx.x; i < k4; i += kQuantThreads) {
    const float4 v = xr[i];
    amax = fmaxf(amax, fmaxf(fmaxf(fabsf(v.x), fabsf(v.y)), fmaxf(fabsf(v.z), fabsf(v.w))));
  }
  amax = block_max(amax, part);
  if (amax == 0.0f) {
    for (int64_t i = threadIdx.x; i < k4; i += kQuantThreads) qr[i] = 0u;
    if (threadIdx.x == 0) x_scale[row] = 0.0f;
    return;
  }
  const float s = amax / 127.0f;
  const float rs = 1.0f / s;
  for (int64_t i = threadIdx.x; i < k4; i += kQuantThreads) qr[i] = quant4(xr[i], s, rs);
  if (threadIdx.x == 0) x_scale[row] = s;
}

}  // namespace

int launch_quantize(const float* x, int64_t m, int64_t k, int8_t* q, float* x_scale,
                    hipStream_t s) {
  const dim3 grid(static_cast<unsigned>(m)), block(kQuantThreads);
  const int64_t nv = ceil_div(k, 4 * kQuantThreads);
  if (nv <= 2) return launch(quantize_rows_reg<2>, grid, block, 0, s, x, k, q, x_scale);
  if (nv <= 4) return launch(quantize_rows_reg<4>, grid, block, 0, s, x, k, q, x_scale);
  if (nv <= 8) return launch(quantize_rows_reg<8>, grid, block, 0, s, x, k, q, x_scale);
  if (nv <= 16) return launch(quantize_rows_reg<16>, grid, block, 0, s, x, k, q, x_scale);
  return launch(quantize_rows, grid, block, 0, s, x, k, q, x_scale);
}

}  // namespace sherry
