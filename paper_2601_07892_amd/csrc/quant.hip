// Per-token int8 activation quantization on the device.
//
// The paper keeps activations in BF16 (weights-only setting, Limitations) but
// its engine accumulates in integers (Appendix A, online phase).  The integer
// inputs are produced here: s = absmax/127, q = clamp(rint(x/s), -127, 127).
// One workgroup per token row; the row is read twice (absmax, then quantize),
// the second time from L2.
#include "sherry_internal.h"

namespace sherry {
namespace {

constexpr int kQuantThreads = 256;

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v = fmaxf(v, __shfl_xor(v, off, 64));
  return v;
}

__device__ __forceinline__ uint32_t quant4(float4 v, float s) {
  float r[4] = {v.x / s, v.y / s, v.z / s, v.w / s};  // IEEE fp32 division
  uint32_t out = 0;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    float t = rintf(r[i]);  // round half to even
    t = fminf(fmaxf(t, -127.0f), 127.0f);
    out |= (static_cast<uint32_t>(static_cast<int>(t)) & 0xFFu) << (8 * i);
  }
  return out;
}

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
  amax = wave_max(amax);
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = amax;
  __syncthreads();
  amax = fmaxf(fmaxf(part[0], part[1]), fmaxf(part[2], part[3]));

  if (amax == 0.0f) {
    for (int64_t i = threadIdx.x; i < k4; i += kQuantThreads) qr[i] = 0u;
    if (threadIdx.x == 0) x_scale[row] = 0.0f;
    return;
  }
  const float s = amax / 127.0f;
  for (int64_t i = threadIdx.x; i < k4; i += kQuantThreads) qr[i] = quant4(xr[i], s);
  if (threadIdx.x == 0) x_scale[row] = s;
}

}  // namespace

int launch_quantize(const float* x, int64_t m, int64_t k, int8_t* q, float* x_scale,
                    hipStream_t s) {
  return launch(quantize_rows, dim3(static_cast<unsigned>(m)), dim3(kQuantThreads), 0,
                     s, x, k, q, x_scale);
}

}  // namespace sherry
