// C ABI entry points: argument validation, M-dispatch, launches.
// Every check happens on the host before anything is enqueued.
#include <cstdlib>

#include <algorithm>
#include <vector>

#include "sherry_internal.h"

namespace sherry {
namespace {
thread_local hipError_t g_last_error = hipSuccess;
}  // namespace
void set_last_error(hipError_t e) { g_last_error = e; }
}  // namespace sherry

using namespace sherry;

namespace {

inline bool aligned(const void* p, uintptr_t a) {
  return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0;
}

inline bool shape_ok(int64_t m, int64_t n, int64_t k) {
  return m >= 1 && n >= 1 && k >= 1 && k % 4 == 0 && m <= SHERRY_MAX_M && n <= SHERRY_MAX_N &&
         k <= SHERRY_MAX_K;
}

inline hipStream_t as_stream(void* s) { return static_cast<hipStream_t>(s); }

int check_fused(const uint8_t* w, const float* x, const float* x_scale, float* y,
                const int32_t* acc, int64_t n, int64_t k) {
  if (!w || !x || !y) return SHERRY_E_INVALID;
  if (!shape_ok(1, n, k) || k > SHERRY_FUSED_MAX_K) return SHERRY_E_SHAPE;
  if (!aligned(w, 16) || !aligned(x, 16) || !aligned(y, 4) || (x_scale && !aligned(x_scale, 4)) ||
      (acc && !aligned(acc, 4)))
    return SHERRY_E_ALIGN;
  return SHERRY_OK;
}

// Largest M the VALU decode kernel serves: up to 4 tokens it is faster than
// the register-decoded MFMA kernel (LLaMA-3.2-3B and 8B-scale projections,
// single launches).
constexpr int64_t kGemvMaxM = 4;
// The register-decoded MFMA kernel takes every product of up to
// kSkinnyMaxLongM tokens and every product with k > n or k >= kSkinnyMinLongK;
// the LDS-tiled kernel keeps the longer products with k <= 2048 <= n (about
// 5% faster on those shapes at 16384 tokens).
constexpr int64_t kSkinnyMinLongK = 3072, kSkinnyMaxLongM = 8192;

int check_product(const uint8_t* w, const int8_t* x, const float* x_scale, float* y,
                  int64_t m, int64_t n, int64_t k, uintptr_t x_align) {
  if (!w || !x || !x_scale || !y) return SHERRY_E_INVALID;
  if (!shape_ok(m, n, k)) return SHERRY_E_SHAPE;
  if (!aligned(w, 16) || !aligned(x, x_align) || !aligned(x_scale, 4) || !aligned(y, 4))
    return SHERRY_E_ALIGN;
  return SHERRY_OK;
}

}  // namespace

extern "C" const char* sherry_status_str(int status) {
  switch (status) {
    case SHERRY_OK: return "ok";
    case SHERRY_E_INVALID: return "invalid argument";
    case SHERRY_E_SHAPE: return "invalid shape";
    case SHERRY_E_NOT_3_4: return "block is not 3:4 (exactly one zero, three +-1)";
    case SHERRY_E_BUFSIZE: return "buffer too small";
    case SHERRY_E_ALIGN: return "misaligned pointer";
    case SHERRY_E_DEVICE: return "device error";
    default: return "unknown status";
  }
}

extern "C" const char* sherry_version(void) { return "sherry 0.1 gfx950"; }

extern "C" const char* sherry_last_error(void) { return hipGetErrorName(g_last_error); }

extern "C" int sherry_quantize_act(const float* x, int64_t m, int64_t k, int8_t* q,
                                   float* x_scale, void* stream) {
  if (!x || !q || !x_scale) return SHERRY_E_INVALID;
  if (!shape_ok(m, 1, k)) return SHERRY_E_SHAPE;
  if (!aligned(x, 16) || !aligned(q, 4) || !aligned(x_scale, 4)) return SHERRY_E_ALIGN;
  return launch_quantize(x, m, k, q, x_scale, as_stream(stream));
}

static_assert(sizeof(sherry_quant_desc) == 40, "sherry_quant_desc layout");

extern "C" int sherry_quantize_act_batched_prepare(sherry_quant_desc* descs, int count,
                                                   int64_t* total_rows, int32_t* max_k) {
  if (!descs || !total_rows || !max_k || count < 1) return SHERRY_E_INVALID;
  int64_t rows = 0;
  int32_t kk = 0;
  for (int i = 0; i < count; ++i) {
    sherry_quant_desc& d = descs[i];
    if (!d.x || !d.q || !d.x_scale) return SHERRY_E_INVALID;
    if (!shape_ok(d.m, 1, d.k)) return SHERRY_E_SHAPE;
    if (!aligned(d.x, 16) || !aligned(d.q, 4) || !aligned(d.x_scale, 4)) return SHERRY_E_ALIGN;
    d.row_begin = static_cast<int32_t>(rows);
    d.reserved = 0;
    rows += d.m;
    if (rows > INT32_MAX) return SHERRY_E_SHAPE;
    if (d.k > kk) kk = d.k;
  }
  *total_rows = rows;
  *max_k = kk;
  return SHERRY_OK;
}

extern "C" int sherry_quantize_act_batched(const sherry_quant_desc* descs_dev, int count,
                                           int64_t total_rows, int32_t max_k, void* stream) {
  if (!descs_dev || count < 1 || total_rows < 1 || total_rows > INT32_MAX)
    return SHERRY_E_INVALID;
  if (max_k < 4 || max_k > SHERRY_MAX_K) return SHERRY_E_SHAPE;
  if (!aligned(descs_dev, 8)) return SHERRY_E_ALIGN;
  return launch_quantize_batched(descs_dev, count, total_rows, max_k, as_stream(stream));
}

extern "C" int sherry_gemm_kernel_for(int64_t m, int64_t n, int64_t k) {
  if (!shape_ok(m, n, k)) return -SHERRY_E_SHAPE;
  if (m <= kGemvMaxM) return SHERRY_KERNEL_GEMV;
  // measured: the register-decoded kernel is as fast or faster on every
  // LLaMA shape up to 8192 tokens and on every k >= 3072 shape; the LDS-tiled
  // kernel keeps the longer, k <= 2048 products (5% faster at 16384 tokens)
  const bool skinny = m <= kSkinnyMaxLongM || k > n || k >= kSkinnyMinLongK;
  return skinny ? SHERRY_KERNEL_SKINNY : SHERRY_KERNEL_MFMA;
}

// The descriptor layouts are part of the ABI (Python and C callers build them).
static_assert(sizeof(sherry_gemv_desc) == 72, "sherry_gemv_desc layout");
static_assert(sizeof(sherry_gemv_f32_desc) == 72, "sherry_gemv_f32_desc layout");
static_assert(sizeof(sherry_gemm_desc) == 80, "sherry_gemm_desc layout");

namespace {
// Product on the chosen kernel (kernel already resolved from AUTO).
int gemm_dispatch(const uint8_t* w, const int8_t* x, const float* x_scale, WScale ws, float* y,
                  int32_t* acc, int64_t m, int64_t n, int64_t k, int kernel, void* stream) {
  if (kernel == SHERRY_KERNEL_AUTO) {
    const int kk = sherry_gemm_kernel_for(m, n, k);
    kernel = kk < 0 ? SHERRY_KERNEL_GEMV : kk;
  }
  if (kernel == SHERRY_KERNEL_GEMV) {
    int st = check_product(w, x, x_scale, y, m, n, k, 4);
    if (st != SHERRY_OK) return st;
    if (m > kGemvMaxM) return SHERRY_E_SHAPE;
    if (acc && !aligned(acc, 4)) return SHERRY_E_ALIGN;
    return launch_gemv_valu(w, x, x_scale, ws, y, acc, m, n, k, as_stream(stream));
  }
  if (kernel == SHERRY_KERNEL_SKINNY) {
    int st = check_product(w, x, x_scale, y, m, n, k, 16);
    if (st != SHERRY_OK) return st;
    if (acc && !aligned(acc, 4)) return SHERRY_E_ALIGN;
    return launch_skinny(w, x, x_scale, ws, y, acc, m, n, k, as_stream(stream));
  }
  if (kernel == SHERRY_KERNEL_MFMA) {
    int st = check_product(w, x, x_scale, y, m, n, k, 16);
    if (st != SHERRY_OK) return st;
    if (acc && !aligned(acc, 4)) return SHERRY_E_ALIGN;
    return launch_gemm_mfma(w, x, x_scale, ws, y, acc, m, n, k, as_stream(stream));
  }
  if (kernel == SHERRY_KERNEL_GEMV_TOK) {
    int st = check_product(w, x, x_scale, y, m, n, k, 4);
    if (st != SHERRY_OK) return st;
    if (!gemv_tok_fits(m, k)) return SHERRY_E_SHAPE;
    if (acc && !aligned(acc, 4)) return SHERRY_E_ALIGN;
    return launch_gemv_tok(w, x, x_scale, ws, nullptr, y, acc, m, n, k, as_stream(stream));
  }
  if (kernel == SHERRY_KERNEL_ALUT) {
    int st = check_product(w, x, x_scale, y, m, n, k, 4);
    if (st != SHERRY_OK) return st;
    if (m != 1 || k > SHERRY_ALUT_MAX_K) return SHERRY_E_SHAPE;
    if (acc && !aligned(acc, 4)) return SHERRY_E_ALIGN;
    return launch_gemv_alut(w, x, x_scale, ws, y, acc, n, k, as_stream(stream));
  }
  return SHERRY_E_INVALID;
}
}  // namespace

extern "C" int sherry_gemm_ex(const uint8_t* w, const int8_t* x, const float* x_scale,
                              float w_scale, float* y, int32_t* acc, int64_t m, int64_t n,
                              int64_t k, int kernel, void* stream) {
  return gemm_dispatch(w, x, x_scale, WScale{nullptr, w_scale}, y, acc, m, n, k, kernel, stream);
}

extern "C" int sherry_gemm_group(const uint8_t* w, const int8_t* x, const float* x_scale,
                                 const float* w_group_scales, float* y, int32_t* acc, int64_t m,
                                 int64_t n, int64_t k, int kernel, void* stream) {
  if (!w_group_scales) return SHERRY_E_INVALID;
  if (!aligned(w_group_scales, 4)) return SHERRY_E_ALIGN;
  if (kernel == SHERRY_KERNEL_AUTO) kernel = m <= kGemvMaxM ? SHERRY_KERNEL_GEMV : SHERRY_KERNEL_SKINNY;
  if (kernel == SHERRY_KERNEL_GEMV) {
    int st = check_product(w, x, x_scale, y, m, n, k, 4);
    if (st != SHERRY_OK) return st;
    if (m > kGemvMaxM) return SHERRY_E_SHAPE;
    if (acc && !aligned(acc, 4)) return SHERRY_E_ALIGN;
    return launch_gemv_group(w, x, x_scale, w_group_scales, y, acc, m, n, k, as_stream(stream));
  }
  if (kernel == SHERRY_KERNEL_GEMV_TOK) {
    int st = check_product(w, x, x_scale, y, m, n, k, 4);
    if (st != SHERRY_OK) return st;
    if (!gemv_tok_fits(m, k)) return SHERRY_E_SHAPE;
    if (acc && !aligned(acc, 4)) return SHERRY_E_ALIGN;
    return launch_gemv_tok(w, x, x_scale, WScale{nullptr, 0.0f}, w_group_scales, y, acc, m, n, k,
                           as_stream(stream));
  }
  if (kernel == SHERRY_KERNEL_SKINNY) {
    int st = check_product(w, x, x_scale, y, m, n, k, 16);
    if (st != SHERRY_OK) return st;
    if (acc && !aligned(acc, 4)) return SHERRY_E_ALIGN;
    return launch_skinny_group(w, x, x_scale, w_group_scales, y, acc, m, n, k,
                               as_stream(stream));
  }
  if (kernel == SHERRY_KERNEL_MFMA) {
    int st = check_product(w, x, x_scale, y, m, n, k, 16);
    if (st != SHERRY_OK) return st;
    if (acc && !aligned(acc, 4)) return SHERRY_E_ALIGN;
    return launch_gemm_mfma_group(w, x, x_scale, w_group_scales, y, acc, m, n, k,
                                  as_stream(stream));
  }
  return SHERRY_E_INVALID;
}

extern "C" int sherry_gemm_channel(const uint8_t* w, const int8_t* x, const float* x_scale,
                                   const float* w_scales, float* y, int32_t* acc, int64_t m,
                                   int64_t n, int64_t k, int kernel, void* stream) {
  if (!w_scales) return SHERRY_E_INVALID;
  if (!aligned(w_scales, 4)) return SHERRY_E_ALIGN;
  return gemm_dispatch(w, x, x_scale, WScale{w_scales, 0.0f}, y, acc, m, n, k, kernel, stream);
}

extern "C" int sherry_gemm(const uint8_t* w, const int8_t* x, const float* x_scale,
                           float w_scale, float* y, int32_t* acc, int64_t m, int64_t n,
                           int64_t k, void* stream) {
  return sherry_gemm_ex(w, x, x_scale, w_scale, y, acc, m, n, k, SHERRY_KERNEL_AUTO, stream);
}

extern "C" int sherry_gemv(const uint8_t* w, const int8_t* x, const float* x_scale,
                           float w_scale, float* y, int32_t* acc, int64_t n, int64_t k,
                           void* stream) {
  return sherry_gemm_ex(w, x, x_scale, w_scale, y, acc, 1, n, k, SHERRY_KERNEL_GEMV, stream);
}

namespace {
// Workgroups of one grouped M = 1 product (same split as the batched kernels).
int64_t gemv_blocks(int64_t n, int64_t k, int target) {
  const int S = gemv_split(static_cast<int>(ceil_div(k, kTileK)), target);
  return ceil_div(ceil_div(n, kTileRows) * S, kGemvWaves);
}
}  // namespace

extern "C" int sherry_gemv_batched_prepare(sherry_gemv_desc* descs, int count,
                                           int64_t* total_blocks) {
  if (!descs || !total_blocks || count < 1) return SHERRY_E_INVALID;
  int64_t blocks = 0;
  for (int i = 0; i < count; ++i) {
    sherry_gemv_desc& d = descs[i];
    int st = check_product(d.w, d.x, d.x_scale, d.y, 1, d.n, d.k, 4);
    if (st != SHERRY_OK) return st;
    if (d.w_scales && d.w_group_scales) return SHERRY_E_INVALID;
    if ((d.acc && !aligned(d.acc, 4)) || (d.w_scales && !aligned(d.w_scales, 4)) ||
        (d.w_group_scales && !aligned(d.w_group_scales, 4)))
      return SHERRY_E_ALIGN;
    d.block_begin = static_cast<int32_t>(blocks);
    blocks += gemv_blocks(d.n, d.k, kGemvTarget);
    if (blocks > INT32_MAX) return SHERRY_E_SHAPE;
  }
  *total_blocks = blocks;
  return SHERRY_OK;
}

extern "C" int sherry_gemv_batched(const sherry_gemv_desc* descs_dev, int count,
                                   int64_t total_blocks, void* stream) {
  if (!descs_dev || count < 1 || total_blocks < 1 || total_blocks > INT32_MAX)
    return SHERRY_E_INVALID;
  if (!aligned(descs_dev, 8)) return SHERRY_E_ALIGN;
  return launch_gemv_batched(descs_dev, count, total_blocks, as_stream(stream));
}

extern "C" int sherry_gemv2(const uint8_t* w2, const int8_t* x, const float* x_scale,
                            float w_scale, float* y, int32_t* acc, int64_t n, int64_t k,
                            void* stream) {
  int st = check_product(w2, x, x_scale, y, 1, n, k, 4);
  if (st != SHERRY_OK) return st;
  if (acc && !aligned(acc, 4)) return SHERRY_E_ALIGN;
  return launch_gemv2(w2, x, x_scale, w_scale, y, acc, n, k, as_stream(stream));
}

extern "C" int sherry_gemv3(const uint8_t* w3, const int8_t* x, const float* x_scale,
                            float w_scale, float* y, int32_t* acc, int64_t n, int64_t k,
                            void* stream) {
  int st = check_product(w3, x, x_scale, y, 1, n, k, 4);
  if (st != SHERRY_OK) return st;
  if (acc && !aligned(acc, 4)) return SHERRY_E_ALIGN;
  return launch_gemv3(w3, x, x_scale, w_scale, y, acc, n, k, as_stream(stream));
}

namespace {
// Grouped launch of M = 1 products on a comparison layout (2 or 3): one
// weight scale per tensor only.
int cmp_batched_prepare(int layout, sherry_gemv_desc* descs, int count, int64_t* total_blocks) {
  if (!descs || !total_blocks || count < 1) return SHERRY_E_INVALID;
  int64_t blocks = 0;
  for (int i = 0; i < count; ++i) {
    sherry_gemv_desc& d = descs[i];
    int st = check_product(d.w, d.x, d.x_scale, d.y, 1, d.n, d.k, 4);
    if (st != SHERRY_OK) return st;
    if (d.w_scales || d.w_group_scales) return SHERRY_E_INVALID;
    if (d.acc && !aligned(d.acc, 4)) return SHERRY_E_ALIGN;
    d.block_begin = static_cast<int32_t>(blocks);
    blocks += cmp_blocks(layout, d.n, d.k);
    if (blocks > INT32_MAX) return SHERRY_E_SHAPE;
  }
  *total_blocks = blocks;
  return SHERRY_OK;
}
int cmp_batched(int layout, const sherry_gemv_desc* descs_dev, int count, int64_t total_blocks,
                void* stream) {
  if (!descs_dev || count < 1 || total_blocks < 1 || total_blocks > INT32_MAX)
    return SHERRY_E_INVALID;
  if (!aligned(descs_dev, 8)) return SHERRY_E_ALIGN;
  return launch_cmp_batched(layout, descs_dev, count, total_blocks, as_stream(stream));
}
}  // namespace

extern "C" int sherry_gemv2_batched_prepare(sherry_gemv_desc* descs, int count,
                                            int64_t* total_blocks) {
  return cmp_batched_prepare(2, descs, count, total_blocks);
}
extern "C" int sherry_gemv2_batched(const sherry_gemv_desc* descs_dev, int count,
                                    int64_t total_blocks, void* stream) {
  return cmp_batched(2, descs_dev, count, total_blocks, stream);
}
extern "C" int sherry_gemv3_batched_prepare(sherry_gemv_desc* descs, int count,
                                            int64_t* total_blocks) {
  return cmp_batched_prepare(3, descs, count, total_blocks);
}
extern "C" int sherry_gemv3_batched(const sherry_gemv_desc* descs_dev, int count,
                                    int64_t total_blocks, void* stream) {
  return cmp_batched(3, descs_dev, count, total_blocks, stream);
}

extern "C" int64_t sherry_stream_read_groups(size_t bytes) { return stream_read_groups(bytes); }

extern "C" int sherry_stream_read(const void* src, size_t bytes, uint32_t* sink, void* stream) {
  if (!src || !sink) return SHERRY_E_INVALID;
  if (bytes == 0 || bytes % 16 != 0) return SHERRY_E_SHAPE;
  if (!aligned(src, 16) || !aligned(sink, 4)) return SHERRY_E_ALIGN;
  return launch_stream_read(src, bytes, sink, as_stream(stream));
}

extern "C" int sherry_gemv_f32(const uint8_t* w, const float* x, float* x_scale, float w_scale,
                               float* y, int32_t* acc, int64_t n, int64_t k, void* stream) {
  int st = check_fused(w, x, x_scale, y, acc, n, k);
  if (st != SHERRY_OK) return st;
  return launch_gemv_f32(w, x, x_scale, WScale{nullptr, w_scale}, y, acc, n, k,
                         as_stream(stream));
}

extern "C" int sherry_gemv_f32_channel(const uint8_t* w, const float* x, float* x_scale,
                                       const float* w_scales, float* y, int32_t* acc, int64_t n,
                                       int64_t k, void* stream) {
  int st = check_fused(w, x, x_scale, y, acc, n, k);
  if (st != SHERRY_OK) return st;
  if (!w_scales) return SHERRY_E_INVALID;
  if (!aligned(w_scales, 4)) return SHERRY_E_ALIGN;
  return launch_gemv_f32(w, x, x_scale, WScale{w_scales, 0.0f}, y, acc, n, k,
                         as_stream(stream));
}

extern "C" int sherry_gemv_f32_group(const uint8_t* w, const float* x, float* x_scale,
                                     const float* w_group_scales, float* y, int32_t* acc,
                                     int64_t n, int64_t k, void* stream) {
  int st = check_fused(w, x, x_scale, y, acc, n, k);
  if (st != SHERRY_OK) return st;
  if (!w_group_scales) return SHERRY_E_INVALID;
  if (!aligned(w_group_scales, 4)) return SHERRY_E_ALIGN;
  return launch_gemv_f32_group(w, x, x_scale, w_group_scales, y, acc, n, k, as_stream(stream));
}

extern "C" int sherry_gemv_f32_batched_prepare(sherry_gemv_f32_desc* descs, int count,
                                               int64_t* total_blocks) {
  if (!descs || !total_blocks || count < 1) return SHERRY_E_INVALID;
  int64_t blocks = 0;
  for (int i = 0; i < count; ++i) {
    sherry_gemv_f32_desc& d = descs[i];
    int st = check_fused(d.w, d.x, d.x_scale, d.y, d.acc, d.n, d.k);
    if (st != SHERRY_OK) return st;
    if (d.w_scales && d.w_group_scales) return SHERRY_E_INVALID;
    if ((d.w_scales && !aligned(d.w_scales, 4)) ||
        (d.w_group_scales && !aligned(d.w_group_scales, 4)))
      return SHERRY_E_ALIGN;
    d.block_begin = static_cast<int32_t>(blocks);
    blocks += ceil_div(ceil_div(d.n, kTileRows) * fused_split(static_cast<int>(ceil_div(d.k, kTileK))),
                       kGemvWaves);
    if (blocks > INT32_MAX) return SHERRY_E_SHAPE;
  }
  *total_blocks = blocks;
  return SHERRY_OK;
}

extern "C" int sherry_gemv_f32_batched(const sherry_gemv_f32_desc* descs_dev, int count,
                                       int64_t total_blocks, void* stream) {
  if (!descs_dev || count < 1 || total_blocks < 1 || total_blocks > INT32_MAX)
    return SHERRY_E_INVALID;
  if (!aligned(descs_dev, 8)) return SHERRY_E_ALIGN;
  return launch_gemv_f32_batched(descs_dev, count, total_blocks, false, as_stream(stream));
}

extern "C" int sherry_gemv_f32_il_batched_prepare(sherry_gemv_f32_desc* descs, int count,
                                                  int64_t* total_blocks) {
  if (!descs || count < 1) return SHERRY_E_INVALID;
  for (int i = 0; i < count; ++i)
    if (descs[i].w_group_scales) return SHERRY_E_INVALID;  // tiled units only
  return sherry_gemv_f32_batched_prepare(descs, count, total_blocks);
}

extern "C" int sherry_gemv_f32_il_batched(const sherry_gemv_f32_desc* descs_dev, int count,
                                          int64_t total_blocks, void* stream) {
  if (!descs_dev || count < 1 || total_blocks < 1 || total_blocks > INT32_MAX)
    return SHERRY_E_INVALID;
  if (!aligned(descs_dev, 8)) return SHERRY_E_ALIGN;
  return launch_gemv_f32_batched(descs_dev, count, total_blocks, true, as_stream(stream));
}

// Block ranges of a grouped launch, numbered in order of decreasing k (ties
// in array order): the workgroups with the longest rows are dispatched first
// and the shorter ones fill in behind them, instead of a few long ones ending
// the launch alone (the LLaMA-3.2-3B step at 16 tokens on lane-interleaved
// weights: 108 us against 121 us in model order).  The kernels find their
// product by its range, so the array keeps the caller's order.
template <class Blocks>
int assign_blocks(sherry_gemm_desc* descs, int count, Blocks nblocks, int64_t* total_blocks) {
  std::vector<int> order(count);
  for (int i = 0; i < count; ++i) order[i] = i;
  std::stable_sort(order.begin(), order.end(),
                   [&](int a, int b) { return descs[a].k > descs[b].k; });
  int64_t blocks = 0;
  for (int i : order) {
    sherry_gemm_desc& d = descs[i];
    const int64_t nb = nblocks(d);
    if (blocks + nb > INT32_MAX) return SHERRY_E_SHAPE;
    d.block_begin = static_cast<int32_t>(blocks);
    d.block_count = static_cast<int32_t>(nb);
    blocks += nb;
  }
  *total_blocks = blocks;
  return SHERRY_OK;
}

extern "C" int sherry_gemm_batched_prepare(sherry_gemm_desc* descs, int count,
                                           int64_t* total_blocks, int32_t* max_m) {
  if (!descs || !total_blocks || !max_m || count < 1) return SHERRY_E_INVALID;
  int32_t mm = 0;
  bool grouped = false;
  for (int i = 0; i < count; ++i) {
    const sherry_gemm_desc& d = descs[i];
    int st = check_product(d.w, d.x, d.x_scale, d.y, d.m, d.n, d.k, 16);
    if (st != SHERRY_OK) return st;
    if ((d.acc && !aligned(d.acc, 4)) || (d.w_scales && !aligned(d.w_scales, 4)) ||
        (d.w_group_scales && !aligned(d.w_group_scales, 4)))
      return SHERRY_E_ALIGN;
    if (d.w_group_scales && (d.w_scales || d.acc)) return SHERRY_E_INVALID;
    if (d.w_group_scales) grouped = true;
    if (d.m > mm) mm = d.m;
  }
  // The launch value *max_m selects the kernel: 1-4 the 4-token matrix-core
  // GEMV (every m <= 4 and every product's activations fit its LDS staging;
  // any scales), 5-16 the 16-token window kernel (every m <= 16; per-group
  // scales with k % 512 == 0, 16-byte aligned), 17 and more the
  // register-decoded kernel (any m, any scales); SHERRY_LAUNCH_GROUPS marks
  // per-group scales.
  bool tok = mm <= 4;
  for (int i = 0; tok && i < count; ++i) tok = gemv_tok_fits(descs[i].m, descs[i].k);
  // the window kernel takes per-group scales of 16-byte aligned rows of a
  // multiple of 4 units (k % 512 == 0)
  bool small = mm <= 16;
  for (int i = 0; small && i < count; ++i) {
    const sherry_gemm_desc& d = descs[i];
    if (d.w_group_scales && (ceil_div(int64_t(d.k), kTileK) % 4 != 0 || !aligned(d.w_group_scales, 16)))
      small = false;
  }
  if (tok || small) {
    const int st = assign_blocks(descs, count, [&](const sherry_gemm_desc& d) {
      return tok ? gemv_tok_blocks(d.n, d.k) : smallm_blocks(d.n);
    }, total_blocks);
    if (st != SHERRY_OK) return st;
    *max_m = (tok ? mm : (mm < 5 ? 5 : mm)) | (grouped ? SHERRY_LAUNCH_GROUPS : 0);
    return SHERRY_OK;
  }
  // otherwise every product runs on the register-decoded kernel in token
  // blocks of the size the largest m selects (per-group scales: 32-token
  // blocks)
  const int32_t sel = grouped && mm > 32 ? 32 : (mm < 17 ? 17 : mm);
  const int64_t tokens = skinny_batched_tokens(sel);
  const int st = assign_blocks(descs, count, [&](const sherry_gemm_desc& d) {
    return int64_t(skinny_blocks(d.n, d.w_group_scales != nullptr)) * ceil_div(d.m, tokens);
  }, total_blocks);
  if (st != SHERRY_OK) return st;
  *max_m = sel | (grouped ? SHERRY_LAUNCH_GROUPS : 0);
  return SHERRY_OK;
}

extern "C" int sherry_gemm_il_batched_prepare(sherry_gemm_desc* descs, int count,
                                              int64_t* total_blocks, int32_t* max_m) {
  if (!descs || !total_blocks || !max_m || count < 1) return SHERRY_E_INVALID;
  int32_t mm = 0;
  for (int i = 0; i < count; ++i) {
    const sherry_gemm_desc& d = descs[i];
    int st = check_product(d.w, d.x, d.x_scale, d.y, d.m, d.n, d.k, 16);
    if (st != SHERRY_OK) return st;
    if (d.m > 16) return SHERRY_E_SHAPE;
    if ((d.acc && !aligned(d.acc, 4)) || (d.w_scales && !aligned(d.w_scales, 4)))
      return SHERRY_E_ALIGN;
    if (d.w_group_scales) return SHERRY_E_INVALID;  // tiled units only
    if (d.m > mm) mm = d.m;
  }
  // launch value 1-4: the 4-token GEMV (every m <= 4, every product's rows fit
  // its LDS staging); 5-16: the 16-token window kernel
  bool tok = mm <= 4;
  for (int i = 0; tok && i < count; ++i) tok = gemv_tok_fits(descs[i].m, descs[i].k);
  const int st = assign_blocks(descs, count, [&](const sherry_gemm_desc& d) {
    return tok ? gemv_tok_blocks(d.n, d.k) : smallm_blocks(d.n);
  }, total_blocks);
  if (st != SHERRY_OK) return st;
  *max_m = tok ? mm : (mm < 5 ? 5 : mm);
  return SHERRY_OK;
}

extern "C" int sherry_gemm_il_batched(const sherry_gemm_desc* descs_dev, int count,
                                      int64_t total_blocks, int32_t max_m, void* stream) {
  if (!descs_dev || count < 1 || total_blocks < 1 || total_blocks > INT32_MAX)
    return SHERRY_E_INVALID;
  if (max_m < 1 || max_m > 16) return SHERRY_E_SHAPE;
  if (!aligned(descs_dev, 8)) return SHERRY_E_ALIGN;
  if (max_m <= 4) return launch_gemv_tok_il_batched(descs_dev, count, total_blocks, as_stream(stream));
  return launch_smallm_il_batched(descs_dev, count, total_blocks, as_stream(stream));
}

extern "C" int sherry_gemm_batched(const sherry_gemm_desc* descs_dev, int count,
                                   int64_t total_blocks, int32_t max_m, void* stream) {
  if (!descs_dev || count < 1 || total_blocks < 1 || total_blocks > INT32_MAX)
    return SHERRY_E_INVALID;
  const bool groups = (max_m & SHERRY_LAUNCH_GROUPS) != 0;
  max_m &= ~SHERRY_LAUNCH_GROUPS;
  if (max_m < 1 || max_m > SHERRY_MAX_M) return SHERRY_E_SHAPE;
  if (!aligned(descs_dev, 8)) return SHERRY_E_ALIGN;
  if (max_m <= 4)
    return launch_gemv_tok_batched(descs_dev, count, total_blocks, groups, as_stream(stream));
  if (max_m <= 16)
    return launch_smallm_batched(descs_dev, count, total_blocks, groups, as_stream(stream));
  return launch_skinny_batched(descs_dev, count, total_blocks, max_m, as_stream(stream));
}

extern "C" int sherry_ternarize_pack(const float* w, int64_t n, int64_t k, uint8_t* packed,
                                     size_t packed_bytes, float* alpha, void* stream) {
  if (!w || !packed) return SHERRY_E_INVALID;
  const size_t need = sherry_packed_bytes(n, k);
  if (need == 0) return SHERRY_E_SHAPE;
  if (packed_bytes < need) return SHERRY_E_BUFSIZE;
  if (!aligned(w, 16) || !aligned(packed, 16) || (alpha && !aligned(alpha, 4)))
    return SHERRY_E_ALIGN;
  return launch_ternarize_pack(w, n, k, packed, alpha, as_stream(stream));
}
