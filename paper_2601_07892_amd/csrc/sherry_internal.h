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
// Unit of the 1.67-bit layout: 64 rows x 96 weights (32 codes of three
// weights per row), stored like a 5-bit unit (1280 bytes).
constexpr int kTileK3 = 96;

constexpr int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Decode kernel work split.  A workgroup has kGemvWaves waves; the
// containers of a 64-row tile are split among S waves of one workgroup,
// S = the smallest power of two with C / S <= target, at most kGemvWaves.
// Up to 16 units per wave (kGemvTarget, kFusedTarget) was measured fastest
// for grouped decode steps, for both the int8 and the fused quantize +
// product kernels: shorter waves (more workgroups, more refills) and longer
// ones (fewer workgroups than the GPU holds) were both slower.
constexpr int kGemvWaves = 8;
constexpr int kGemvTarget = 16;
constexpr int kFusedTarget = 16;
// Longest activation row of the fused quantize + product kernels (the
// quantized row is held in LDS); equals SHERRY_FUSED_MAX_K.
constexpr int kFusedMaxK = SHERRY_FUSED_MAX_K;
__host__ __device__ constexpr int gemv_split(int C, int target = kGemvTarget) {
  int s = 1;
  while (s < kGemvWaves && C > s * target) s *= 2;
  return s;
}

// Split of the grouped fused kernel: a row of up to 2 * kFusedTarget units
// stays in one wave (LLaMA-3.2-3B steps, whose k = 3072 products have 24
// units, measured 2.4% faster than with those split in two), longer rows as
// gemv_split.
__host__ __device__ constexpr int fused_split(int C) {
  return C <= 2 * kFusedTarget ? 1 : gemv_split(C, kFusedTarget);
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

// Per-token activation quantization, shared by the quantize kernel and the
// fused quantize + product kernel so that both take identical decisions:
// max over a wave, and four values to int8 with s = absmax / 127:
// q = clamp(rint(x / s), -127, 127), IEEE fp32 division, ties to even.
__device__ __forceinline__ float wave_max_f32(float v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v = fmaxf(v, __shfl_xor(v, off, 64));
  return v;
}

// rint(x / s) with the IEEE quotient, mostly without dividing.  rs = 1 / s
// (correctly rounded) and t = x * rs are each within half an ulp, so t is
// within 2^-23 * |x / s| <= 1.6e-5 of the exact quotient (|x / s| <= 127 +
// a few ulps), and the rounded quotient within 2^-18 of it.  When t lies
// at least 2^-13 from every half-integer, the rounded quotient is in the
// same unit interval and rounds to the same integer as t; otherwise (also
// for a non-finite t, e.g. a tiny s whose reciprocal overflows) the
// division itself decides.
__device__ __forceinline__ float round_quotient(float x, float s, float rs) {
  const float t = x * rs;
  const float k = rintf(t);
  const float d = fabsf(t - k);  // exact: distance to the nearest integer
  if (!(d <= 0.5f - 0x1p-13f)) return rintf(x / s);
  return k;
}

__device__ __forceinline__ uint32_t quant4(float4 v, float s, float rs) {
  const float r[4] = {round_quotient(v.x, s, rs), round_quotient(v.y, s, rs),
                      round_quotient(v.z, s, rs), round_quotient(v.w, s, rs)};
  uint32_t out = 0;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const float t = fminf(fmaxf(r[i], -127.0f), 127.0f);
    out |= (static_cast<uint32_t>(static_cast<int>(t)) & 0xFFu) << (8 * i);
  }
  return out;
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

// Descriptor of a grouped launch whose block range [block_begin, block_begin
// + block_count) holds block blk (the grouped prepares number the products'
// blocks longest rows first, so the ranges follow no order of the array):
// 64 descriptors per ballot round.  -1 if none does (a grid larger than the
// prepared total): the workgroup then has no work.
template <class Desc>
__device__ __forceinline__ int find_block_desc(const Desc* descs, int count, int32_t blk) {
  const int lane = threadIdx.x & 63;
  for (int base = 0; base < count; base += 64) {
    const int i = base + lane;
    bool hit = false;
    if (i < count) {
      const int32_t b0 = as_global(descs)[i].block_begin;
      const int32_t nb = as_global(descs)[i].block_count;
      hit = b0 <= blk && blk - b0 < nb;
    }
    const uint64_t m = __ballot(hit);
    if (m) return __builtin_amdgcn_readfirstlane(base + static_cast<int>(__builtin_ctzll(m)));
  }
  return -1;
}

// Weight scale of output row n: one per tensor, or, when rows is set, one
// per output channel ([T alpha]_ij = T_ij alpha_j, the footnote to Eq. 2).
// A wave's run of n consecutive weight units of B bytes each, from base.
// Unit c is read through a buffer resource over that unit alone, and an
// empty one for c >= n: its loads then return zeros without touching memory,
// since the range check applies to the per-lane offset (soffset is left at
// zero).  Reads past the run can so be issued on every path, which keeps the
// compiler's waits on exact load counts; the resource costs scalar
// instructions only.
struct UnitRun {
  const uint8_t* base;
  int n;
  template <int B>
  __device__ __forceinline__ __amdgpu_buffer_rsrc_t unit(int c) const {
    const bool in = c < n;
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t*>(base) + int64_t(in ? c : 0) * B,
                                             0, in ? B : 0, kBufferWord3);
  }
};

// Unit c of a run in the tiled layout: 16-byte head at lane*16, 4-byte tail
// at kHeadBytes + lane*4.
__device__ __forceinline__ void load_unit(uint32_t (&d)[5], const UnitRun& run, int c, int lane) {
  const __amdgpu_buffer_rsrc_t r = run.unit<kUnitBytes>(c);
  const u32x4 h = __builtin_amdgcn_raw_buffer_load_b128(r, 16 * lane, 0, kLoadStream);
  d[0] = h.x;
  d[1] = h.y;
  d[2] = h.z;
  d[3] = h.w;
  d[4] = __builtin_amdgcn_raw_buffer_load_b32(r, kHeadBytes + 4 * lane, 0, kLoadStream);
}

struct WScale {
  const float* rows;
  float tensor;
  __device__ __forceinline__ float at(int64_t n) const {
    return rows ? as_global(rows)[n] : tensor;
  }
};

// ---- host-side launchers (each returns a sherry_status) -------------------

int launch_quantize(const float* x, int64_t m, int64_t k, int8_t* q,
                    float* x_scale, hipStream_t s);
// Every row of a prepared descriptor array (total_rows workgroups); max_k
// selects how rows are held (registers or two passes).
int launch_quantize_batched(const sherry_quant_desc* descs, int count, int64_t total_rows,
                            int64_t max_k, hipStream_t s);

int launch_gemv_valu(const uint8_t* w, const int8_t* x, const float* x_scale,
                     WScale ws, float* y, int32_t* acc, int64_t m,
                     int64_t n, int64_t k, hipStream_t s);

// Activation-table product for one token (k <= SHERRY_ALUT_MAX_K).
int launch_gemv_alut(const uint8_t* w, const int8_t* x, const float* x_scale, WScale ws,
                     float* y, int32_t* acc, int64_t n, int64_t k, hipStream_t s);

// Up to four tokens on the matrix cores, activations staged in LDS
// (m * ceil(k/128) * 128 <= 32768 bytes, gemv_tok_fits): single and grouped
// launches, per-tensor, per-channel or (gs != nullptr) per-group scales;
// gemv_tok_blocks is one product's workgroup count in a grouped launch.
bool gemv_tok_fits(int64_t m, int64_t k);
int launch_gemv_tok(const uint8_t* w, const int8_t* x, const float* x_scale, WScale ws,
                    const float* gs, float* y, int32_t* acc, int64_t m, int64_t n, int64_t k,
                    hipStream_t s);
int64_t gemv_tok_blocks(int64_t n, int64_t k);
// The same products on lane-interleaved weights (no per-group scales).
int launch_gemv_tok_il_batched(const sherry_gemm_desc* descs, int count, int64_t total_blocks,
                               hipStream_t s);
int launch_gemv_tok_batched(const sherry_gemm_desc* descs, int count, int64_t total_blocks,
                            bool groups, hipStream_t s);

// Up to 16 tokens on the matrix cores, weights as loaded, activations
// staged per K window (grouped launches): one product's workgroup count, and
// the launch.
int launch_smallm_il_batched(const sherry_gemm_desc* descs, int count, int64_t total_blocks,
                             hipStream_t s);
int64_t smallm_blocks(int64_t n);
int launch_smallm_batched(const sherry_gemm_desc* descs, int count, int64_t total_blocks,
                          bool groups, hipStream_t s);

int skinny_blocks(int64_t n, bool group_scales = false);
int skinny_batched_tokens(int max_m);
int launch_skinny(const uint8_t* w, const int8_t* x, const float* x_scale, WScale ws,
                  float* y, int32_t* acc, int64_t m, int64_t n, int64_t k, hipStream_t s);
int launch_skinny_batched(const sherry_gemm_desc* descs, int count, int64_t total_blocks,
                          int max_m, hipStream_t s);
int launch_gemv_batched(const sherry_gemv_desc* descs, int count,
                        int64_t total_blocks, hipStream_t s);
int launch_gemv_f32(const uint8_t* w, const float* x, float* x_scale, WScale ws, float* y,
                    int32_t* acc, int64_t n, int64_t k, hipStream_t s);
// il: lane-interleaved units (sherry_pack_il; no per-group scales).
int launch_gemv_f32_batched(const sherry_gemv_f32_desc* descs, int count, int64_t total_blocks,
                            bool il, hipStream_t s);
// Per-group weight scales gs: fp32 [n][ceil(k/128)] (one per 128 weights of
// a row).
int launch_gemv_group(const uint8_t* w, const int8_t* x, const float* x_scale, const float* gs,
                      float* y, int32_t* acc, int64_t m, int64_t n, int64_t k, hipStream_t s);
int launch_gemv_f32_group(const uint8_t* w, const float* x, float* x_scale, const float* gs,
                          float* y, int32_t* acc, int64_t n, int64_t k, hipStream_t s);
int launch_skinny_group(const uint8_t* w, const int8_t* x, const float* x_scale, const float* gs,
                        float* y, int32_t* acc, int64_t m, int64_t n, int64_t k, hipStream_t s);

// MFMA tile configuration chosen for an m x n product: 0 skinny (32 x 256),
// 1 small (128 x 128), 2 mid (128 x 256), 3 large (256 x 256).
int gemm_config_for(int64_t m, int64_t n);
int launch_gemm_mfma_group(const uint8_t* w, const int8_t* x, const float* x_scale,
                           const float* gs, float* y, int32_t* acc, int64_t m, int64_t n,
                           int64_t k, hipStream_t s);
int launch_gemm_mfma(const uint8_t* w, const int8_t* x, const float* x_scale,
                     WScale ws, float* y, int32_t* acc, int64_t m,
                     int64_t n, int64_t k, hipStream_t s);

// Comparison layouts (M = 1, one weight scale per tensor): 2-bit and
// 1.67-bit.  cmp_blocks(layout, n, k) is the workgroup count of one product
// (layout 2 or 3); launch_cmp_batched runs a prepared descriptor array.
int launch_gemv2(const uint8_t* w2, const int8_t* x, const float* x_scale,
                 float w_scale, float* y, int32_t* acc, int64_t n, int64_t k,
                 hipStream_t s);
int launch_gemv3(const uint8_t* w3, const int8_t* x, const float* x_scale,
                 float w_scale, float* y, int32_t* acc, int64_t n, int64_t k,
                 hipStream_t s);
int64_t cmp_blocks(int layout, int64_t n, int64_t k);
int launch_cmp_batched(int layout, const sherry_gemv_desc* descs, int count,
                       int64_t total_blocks, hipStream_t s);

int launch_stream_read(const void* src, size_t bytes, uint32_t* sink,
                       hipStream_t s);

int launch_ternarize_pack(const float* w, int64_t n, int64_t k, uint8_t* out, float* alpha,
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
