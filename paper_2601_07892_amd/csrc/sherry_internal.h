// Internal declarations of the Sherry gfx950 library (not part of the ABI).
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>
#include <tuple>
#include <utility>

#include "../../include/sherry.h"

namespace sherry {

// Unit of the packed 5-bit layout: 64 rows x 128 weights (32 codes per row).
constexpr int kTileRows = 64;
constexpr int kTileK = 128;
constexpr int kUnitBytes = 1280;   // 64 * 20
constexpr int kHeadBytes = 1024;   // 64 rows * 16 bytes
// Unit of the 2-bit layout: 64 rows x 64 weights, 16 bytes per row.
constexpr int kTileK2 = 64;
constexpr int kUnit2Bytes = 1024;

constexpr int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Decode kernel work split.  A workgroup has kGemvWaves waves; the
// containers of a 64-row tile are split among S waves of one workgroup,
// S = the smallest power of two with C / S <= kGemvTarget, at most
// kGemvWaves.  Short waves keep many workgroups queued behind the resident
// ones, so a CU that finishes early is refilled instead of idling.
constexpr int kGemvWaves = 8;
constexpr int kGemvTarget = 8;
__host__ __device__ constexpr int gemv_split(int C) {
  int s = 1;
  while (s < kGemvWaves && C > s * kGemvTarget) s *= 2;
  return s;
}

// Decoded weights of a 5-bit code as a little-endian int8x4 word (byte p =
// weight at block position p: +1 -> 0x01, -1 -> 0xFF, 0 -> 0x00).  The code
// is z | s0<<2 | s1<<3 | s2<<4: z = zero position, si = sign bit of the i-th
// non-zero in ascending position (1 = negative).
__host__ __device__ constexpr uint32_t decode_word(uint32_t code) {
  const uint32_t z = code & 3u;
  const uint32_t s = code >> 2;
  uint32_t word = 0;
  int i = 0;
  for (uint32_t p = 0; p < 4; ++p) {
    if (p == z) continue;
    const uint32_t byte = ((s >> i) & 1u) ? 0xFFu : 0x01u;
    word |= byte << (8 * p);
    ++i;
  }
  return word;
}

// Byte offset (code*4) in the 32-entry table of code j (0..31) of a row's
// 160-bit stream held in d[0..4] (stream bit b = bit b%32 of d[b/32]): one
// funnel shift and one mask.
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

// Address-space views of device pointers.  Pointers read from memory (e.g.
// from a descriptor array) are generic to the compiler; these casts let it
// emit global loads, and scalar loads for data that is read-only during the
// kernel and addressed uniformly across the wave (constant address space).
// (The host compilation pass of the same source sees no address spaces.)
#if defined(__HIP_DEVICE_COMPILE__)
#define SHERRY_GLOBAL __attribute__((address_space(1)))
#define SHERRY_CONST __attribute__((address_space(4)))
#else
#define SHERRY_GLOBAL
#define SHERRY_CONST
#endif

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Word 3 of a raw buffer resource on gfx9-family GPUs (untyped 32-bit data,
// no swizzle): address = base + voffset + soffset + imm, bounded by the
// resource's byte count.
constexpr int kBufferWord3 = 0x00020000;
// Cache-policy operand of buffer loads: non-temporal.  The packed weights
// are read exactly once per product; streaming them as non-temporal lifts
// sustained read bandwidth from about 6.3 to 7.1 TB/s on MI355X.
constexpr int kLoadStream = 2;

template <class T>
__device__ __forceinline__ const SHERRY_CONST T* as_const(const T* p) {
  return (const SHERRY_CONST T*)(p);
}
template <class T>
__device__ __forceinline__ const SHERRY_GLOBAL T* as_global(const T* p) {
  return (const SHERRY_GLOBAL T*)(p);
}
template <class T>
__device__ __forceinline__ SHERRY_GLOBAL T* as_global_mut(T* p) {
  return (SHERRY_GLOBAL T*)(p);
}

// ---- host-side launchers (each returns a sherry_status) -------------------

int launch_quantize(const float* x, int64_t m, int64_t k, int8_t* q,
                    float* x_scale, hipStream_t s);

int launch_gemv_valu(const uint8_t* w, const int8_t* x, const float* x_scale,
                     float w_scale, float* y, int32_t* acc, int64_t m,
                     int64_t n, int64_t k, hipStream_t s);

int launch_gemv_batched(const sherry_gemv_desc* descs, int count,
                        int64_t total_blocks, hipStream_t s);

// MFMA tile configuration chosen for an m x n product: 0 skinny (32 x 256),
// 1 small (128 x 128), 2 mid (128 x 256), 3 large (256 x 256).
int gemm_config_for(int64_t m, int64_t n);
int launch_gemm_mfma(const uint8_t* w, const int8_t* x, const float* x_scale,
                     float w_scale, float* y, int32_t* acc, int64_t m,
                     int64_t n, int64_t k, hipStream_t s);

int launch_gemv2(const uint8_t* w2, const int8_t* x, const float* x_scale,
                 float w_scale, float* y, int32_t* acc, int64_t n, int64_t k,
                 hipStream_t s);

int launch_stream_read(const void* src, size_t bytes, uint32_t* sink,
                       hipStream_t s);
int64_t stream_read_groups(size_t bytes);

// Records the HIP error of the calling thread's last failed library call
// (read back through sherry_last_error).
void set_last_error(hipError_t e);

// Launches `kernel` through hipLaunchKernel, which returns the status of this
// launch itself (not an error left behind by earlier, unrelated HIP calls).
template <typename... KArgs, typename... Args>
int launch(void (*kernel)(KArgs...), dim3 grid, dim3 block, size_t shmem, hipStream_t s,
           Args&&... args) {
  std::tuple<KArgs...> vals(std::forward<Args>(args)...);
  void* ptrs[sizeof...(KArgs)];
  std::apply([&](auto&... v) {
    int i = 0;
    ((ptrs[i++] = static_cast<void*>(&v)), ...);
  }, vals);
  const hipError_t e =
      hipLaunchKernel(reinterpret_cast<const void*>(kernel), grid, block, ptrs, shmem, s);
  if (e != hipSuccess) {
    set_last_error(e);
    return SHERRY_E_DEVICE;
  }
  return SHERRY_OK;
}

}  // namespace sherry
