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

// One row x[0..k) -> q, *scale, by the whole workgroup.  NV > 0: rows of up
// to NV*1024 values, read once into registers (NV float4 per thread),
// reduced and quantized from registers.  NV = 0: any row length, two passes
// over the row (the second from cache).
template <int NV>
__device__ __forceinline__ void quantize_row(const float* x, int64_t k, int8_t* q, float* scale,
                                             float* part) {
  const float4* xr = reinterpret_cast<const float4*>(x);
  uint32_t* qr = reinterpret_cast<uint32_t*>(q);
  if constexpr (NV > 0) {
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
    if (threadIdx.x == 0) *scale = (amax == 0.0f) ? 0.0f : s;
  } else {
    const int64_t k4 = k >> 2;
    float amax = 0.0f;
    for (int64_t i = threadIdx.x; i < k4; i += kQuantThreads) {
      const float4 v = xr[i];
      amax = fmaxf(amax, fmaxf(fmaxf(fabsf(v.x), fabsf(v.y)), fmaxf(fabsf(v.z), fabsf(v.w))));
    }
    amax = block_max(amax, part);
    if (amax == 0.0f) {
      for (int64_t i = threadIdx.x; i < k4; i += kQuantThreads) qr[i] = 0u;
      if (threadIdx.x == 0) *scale = 0.0f;
      return;
    }
    const float s = amax / 127.0f;
    const float rs = 1.0f / s;
    for (int64_t i = threadIdx.x; i < k4; i += kQuantThreads) qr[i] = quant4(xr[i], s, rs);
    if (threadIdx.x == 0) *scale = s;
  }
}

template <int NV>
__global__ __launch_bounds__(kQuantThreads) void quantize_rows_kernel(
    const float* __restrict__ x, int64_t k, int8_t* __restrict__ q,
    float* __restrict__ x_scale) {
  __shared__ float part[kQuantThreads / 64];
  const int64_t row = blockIdx.x;
  quantize_row<NV>(x + row * k, k, q + row * k, x_scale + row, part);
}

// Every row of every matrix of a descriptor array, one workgroup per row.
template <int NV>
__global__ __launch_bounds__(kQuantThreads) void quantize_batched_kernel(
    const sherry_quant_desc* __restrict__ descs, int count) {
  __shared__ float part[kQuantThreads / 64];
  const int32_t blk = static_cast<int32_t>(blockIdx.x);
  // last descriptor with row_begin <= blk (a prefix: row_begin increases)
  const int lane = threadIdx.x & 63;
  int lo = 0;
  for (int base = 0; base < count; base += 64) {
    const int i = base + lane;
    const bool ok = i < count && as_global(descs)[i].row_begin <= blk;
    const int len = __popcll(__ballot(ok));
    lo = base + len - 1;
    if (len < 64) break;
  }
  lo = __builtin_amdgcn_readfirstlane(lo);
  const sherry_quant_desc& d = descs[lo];
  const int64_t row = blk - d.row_begin, k = d.k;
  quantize_row<NV>(d.x + row * k, k, d.q + row * k, d.x_scale + row, part);
}

// Register-held rows up to NV*1024 values; 0 = two passes.
int quant_nv(int64_t k) {
  const int64_t nv = ceil_div(k, 4 * kQuantThreads);
  return nv <= 2 ? 2 : nv <= 4 ? 4 : nv <= 8 ? 8 : nv <= 16 ? 16 : 0;
}

}  // namespace

int launch_quantize(const float* x, int64_t m, int64_t k, int8_t* q, float* x_scale,
                    hipStream_t s) {
  const dim3 grid(static_cast<unsigned>(m)), block(kQuantThreads);
  switch (quant_nv(k)) {
    case 2: return launch(quantize_rows_kernel<2>, grid, block, 0, s, x, k, q, x_scale);
    case 4: return launch(quantize_rows_kernel<4>, grid, block, 0, s, x, k, q, x_scale);
    case 8: return launch(quantize_rows_kernel<8>, grid, block, 0, s, x, k, q, x_scale);
    case 16: return launch(quantize_rows_kernel<16>, grid, block, 0, s, x, k, q, x_scale);
    default: return launch(quantize_rows_kernel<0>, grid, block, 0, s, x, k, q, x_scale);
  }
}

int launch_quantize_batched(const sherry_quant_desc* descs, int count, int64_t total_rows,
                            int64_t max_k, hipStream_t s) {
  const dim3 grid(static_cast<unsigned>(total_rows)), block(kQuantThreads);
  switch (quant_nv(max_k)) {
    case 2: return launch(quantize_batched_kernel<2>, grid, block, 0, s, descs, count);
    case 4: return launch(quantize_batched_kernel<4>, grid, block, 0, s, descs, count);
    case 8: return launch(quantize_batched_kernel<8>, grid, block, 0, s, descs, count);
    case 16: return launch(quantize_batched_kernel<16>, grid, block, 0, s, descs, count);
    default: return launch(quantize_batched_kernel<0>, grid, block, 0, s, descs, count);
  }
}

}  // namespace sherry
