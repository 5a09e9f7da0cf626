/*
 * sherry.h -- C ABI of the MI355X (gfx950) library for the Sherry 3:4 sparse
 * ternary product (arXiv 2601.07892).
 *
 * The library computes the inference-time product of Eq. 2,
 *
 *     Y = X T alpha,
 *
 * where T (N x K here: row n is the paper's output channel j, K its d_in)
 * has values in {-1, 0, +1} and satisfies the 3:4 constraint of Eq. 3: in
 * every block of 4 consecutive weights along K exactly one is zero.  Each
 * block is stored as one 5-bit code (Sec. 3.1, point 3: C(4,3)*2^3 = 32
 * states), 1.25 bits per weight (offline packing phase, Appendix A).  X is
 * int8 with one fp32 scale per token, alpha a per-tensor fp32 scale, and the
 * product is accumulated exactly in int32 (online phase, Appendix A):
 *
 *     acc[m][n] = sum_k X[m][k] * T[n][k]                 (exact, int32)
 *     y[m][n]   = float(acc[m][n]) * (x_scale[m] * w_scale)  (fp32, RNE)
 *
 * Conventions for every call:
 *  - Every entry point returns a sherry_status (0 = SHERRY_OK).  Arguments are
 *    validated on the host before anything is enqueued; on any error nothing
 *    runs and output buffers are untouched.
 *  - "host" pointers are ordinary CPU memory; "device" pointers are HIP device
 *    memory of the current device.  The caller owns and frees every buffer;
 *    the library allocates nothing and keeps no mutable global state apart
 *    from a per-thread record of the last HIP error, so calls from several
 *    threads are safe (calls that write the same buffers race).
 *  - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *    Device calls are asynchronous: they enqueue kernels and return.  Launch
 *    failures return SHERRY_E_DEVICE; faults surface at the next sync.
 *  - Sizes are in elements unless named *_bytes.  All matrices are row-major.
 *
 * Packed 5-bit tiled layout (what sherry_pack writes and the products read):
 *  - code of a block = z | s0<<2 | s1<<3 | s2<<4, z = position (0..3, lowest
 *    K first) of the zero, si = 1 when the i-th non-zero (ascending position)
 *    is -1.  code ^ 0x1C negates the block (the mirror pairs of Appendix C).
 *  - rows padded to Np = ceil(N/64)*64, K to Kp = ceil(K/128)*128; padding
 *    codes are zero bits.
 *  - unit (r, c) = 64 rows x 128 weights = 1280 bytes at (r*Kp/128 + c)*1280.
 *    Row i of the unit is a 160-bit little-endian stream, code j (weights
 *    128c+4j..+3) at bits [5j, 5j+5); stream bits 0..127 are the 16 bytes at
 *    16*i, bits 128..159 the 4 bytes at 1024 + 4*i.
 *  Total size: Np * Kp * 5 / 32 bytes (exactly 5NK/32 when 64 | N, 128 | K).
 */
#ifndef SHERRY_H_
#define SHERRY_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum sherry_status {
  SHERRY_OK = 0,
  SHERRY_E_INVALID = 1,  /* null pointer or an argument out of its domain   */
  SHERRY_E_SHAPE = 2,    /* m, n or k < 1, k % 4 != 0, or beyond the limits */
  SHERRY_E_NOT_3_4 = 3,  /* a block of T is not exactly one 0 and three +-1 */
  SHERRY_E_BUFSIZE = 4,  /* a caller buffer is smaller than required        */
  SHERRY_E_ALIGN = 5,    /* a device pointer is not aligned as documented   */
  SHERRY_E_DEVICE = 6    /* a HIP call or kernel launch failed              */
} sherry_status;

/* Largest accepted K: |acc| <= 127 * 3K/4 must stay exact in fp32 (< 2^24)
 * and in int32; 2^24 / (128 * 3/4) = 174762, rounded down to 128 | K. */
#define SHERRY_MAX_K 174720
/* Largest accepted N and M (grid limits; far above any LLM layer). */
#define SHERRY_MAX_N (1LL << 26)
#define SHERRY_MAX_M (1LL << 24)
/* Longest activation row of the fused quantize + product calls (the
 * quantized row is staged on chip). */
#define SHERRY_FUSED_MAX_K 32768

/* Kernel selectors for sherry_gemm_ex (see sherry_gemm_kernel_for for the
 * automatic choice). */
#define SHERRY_KERNEL_AUTO 0
#define SHERRY_KERNEL_GEMV 1 /* VALU decode + dot4 per token, M <= 4         */
#define SHERRY_KERNEL_MFMA 2 /* decode to int8 tiles in LDS + int8 MFMA      */
#define SHERRY_KERNEL_SKINNY 3 /* decode in registers + int8 MFMA, any M     */
/* Activation lookup tables, M = 1, k <= SHERRY_ALUT_MAX_K: the table        */
/* direction of the paper's CPU engine (16 dot products per block of 4       */
/* activations, 4-bit index + sign bit per code; Sec. 3.1, Appendix A), a    */
/* comparison point for SHERRY_KERNEL_GEMV.  Never chosen automatically.     */
#define SHERRY_KERNEL_ALUT 4
/* Decode in registers + one int8 MFMA per 4-code chunk for up to 4 tokens  */
/* (the activations staged in LDS): m <= 4 and m*ceil(k/128)*128 <= 32768.  */
#define SHERRY_KERNEL_GEMV_TOK 5
#define SHERRY_ALUT_MAX_K 8192

/* Static string for a status code (never NULL). */
const char* sherry_status_str(int status);

/* Library version string, e.g. "sherry 0.1 gfx950". */
const char* sherry_version(void);

/* Name of the HIP error behind the calling thread's most recent
 * SHERRY_E_DEVICE ("hipSuccess" if none).  Static string, never NULL. */
const char* sherry_last_error(void);

/* ---------------------------------------------------------------------- */
/* Offline packing (Appendix A, offline phase).  Host only.               */
/* ---------------------------------------------------------------------- */

/* Bytes of the packed 5-bit tiled layout for an n x k ternary matrix; 0 if
 * n < 1, k < 1, k % 4 != 0, n > SHERRY_MAX_N or k > SHERRY_MAX_K. */
size_t sherry_packed_bytes(int64_t n, int64_t k);

/* Packs T (host, int8 [n][k] row-major, values in {-1,0,1}, exactly one zero
 * in every 4-block along k) into out (host, out_bytes >=
 * sherry_packed_bytes(n, k)); the first sherry_packed_bytes(n, k) bytes are
 * written, padding included.  On SHERRY_E_NOT_3_4 the flat index n*(k/4)+b
 * of the first offending block is stored to *bad_block when bad_block is not
 * NULL (else it is left alone), and out is unspecified.  Uses host threads. */
int sherry_pack(const int8_t* t, int64_t n, int64_t k, uint8_t* out,
                size_t out_bytes, int64_t* bad_block);

/* Exact inverse of sherry_pack: reads packed (host, packed_bytes >=
 * sherry_packed_bytes(n, k)) and writes t_out (host, int8 [n][k]). */
int sherry_unpack(const uint8_t* packed, size_t packed_bytes, int64_t n,
                  int64_t k, int8_t* t_out);

/* Lane-interleaved layout: the same 5-bit codes, units and byte size as the
 * tiled layout, with the codes of each unit assigned to lanes for the int8
 * matrix cores.  Container l = 16b + t of a unit (head bytes 16l..16l+15,
 * tail bytes 1024+4l..1024+4l+3, code j at stream bits [5j, 5j+5) as in the
 * tiled layout) holds as code j = 4(2g + p) + c the code of row 16g + t of
 * the unit and of its block 16p + 4b + c (weights 4(16p+4b+c) .. +3 of the
 * unit's 128), for g, b in 0..3, p in 0..1, c in 0..3.  So a lane's codes
 * 4(2g+p) .. 4(2g+p)+3 are row 16g + t's 16 weights of chunk 4p + b.
 * sherry_pack_il / sherry_unpack_il: as sherry_pack / sherry_unpack, in this
 * layout.  Read by the *_il products only. */
int sherry_pack_il(const int8_t* t, int64_t n, int64_t k, uint8_t* out,
                   size_t out_bytes, int64_t* bad_block);
int sherry_unpack_il(const uint8_t* packed, size_t packed_bytes, int64_t n,
                     int64_t k, int8_t* t_out);

/* Device: rewrites tiled units (tiled, e.g. from sherry_ternarize_pack) as
 * lane-interleaved units (il), both sherry_packed_bytes(n, k) bytes,
 * 16-byte aligned, and not overlapping (overlapping buffers give undefined
 * results; only tiled == il is detected); one wave per unit.
 * SHERRY_E_SHAPE as sherry_packed_bytes, SHERRY_E_INVALID for NULL or
 * tiled == il, SHERRY_E_ALIGN for a misaligned buffer. */
int sherry_interleave(const uint8_t* tiled, uint8_t* il, int64_t n, int64_t k, void* stream);

/* Sparse-AbsMean ternarization and packing on the GPU (Eq. 4, Eq. 5), the
 * step that turns full-precision weights into the packed layout.
 * w: device, fp32 [n][k] row-major (row = output channel, blocks of 4 along
 * k), 16-byte aligned, finite values.  In each block of 4 the smallest |w|
 * becomes 0 (ties: the lowest position) and the other three their sign (+1
 * for a kept zero).  packed: device, packed_bytes >= sherry_packed_bytes(n,
 * k), 16-byte aligned; receives exactly the bytes sherry_pack writes for that
 * ternary matrix.  alpha: device, fp32 [n], 4-byte aligned, or NULL;
 * receives Eq. 5 per output channel, the mean |w| over the row's kept
 * weights, summed in fp64 (the summation order differs from a sequential
 * sum, so the fp32 result can differ from one by a unit in the last place).
 * Enqueued on stream; returns SHERRY_E_SHAPE / _BUFSIZE / _ALIGN /
 * _INVALID before enqueuing anything. */
int sherry_ternarize_pack(const float* w, int64_t n, int64_t k, uint8_t* packed,
                          size_t packed_bytes, float* alpha, void* stream);

/* ---------------------------------------------------------------------- */
/* Activation quantization (the integer inputs of the online phase).       */
/* ---------------------------------------------------------------------- */

/* Per-token int8 quantization on the device.  x (device, fp32 [m][k], 16-byte
 * aligned, finite values) -> q (device, int8 [m][k], 4-byte aligned) and
 * x_scale (device, fp32 [m]):  s = max_k |x| / 127 (fp32 division);
 * q = clamp(rint(x / s), -127, 127) with round-half-to-even; an all-zero row
 * gives s = 0 and q = 0.  The paper does not specify activation quantization
 * (its weights-only setting keeps BF16 activations, Limitations); this is
 * the int8 per-token reading of the integer accumulation of Appendix A. */
int sherry_quantize_act(const float* x, int64_t m, int64_t k, int8_t* q,
                        float* x_scale, void* stream);

/* Many activation matrices in one launch (e.g. the inputs of every linear
 * of a model step), each quantized exactly as sherry_quantize_act does. */
typedef struct sherry_quant_desc {
  const float* x;      /* device, fp32 [m][k], 16-byte aligned             */
  int8_t* q;           /* device, int8 [m][k], 4-byte aligned              */
  float* x_scale;      /* device, fp32 [m]                                 */
  int32_t m, k;        /* m >= 1; k >= 4, k % 4 == 0, k <= SHERRY_MAX_K    */
  int32_t row_begin;   /* written by sherry_quantize_act_batched_prepare   */
  int32_t reserved;    /* set to 0                                         */
} sherry_quant_desc;

/* Host: validates descs[0..count) (count >= 1), fills each row_begin (the
 * first row of that matrix in the launch), *total_rows (all rows) and
 * *max_k (the longest row); pass both to sherry_quantize_act_batched. */
int sherry_quantize_act_batched_prepare(sherry_quant_desc* descs, int count,
                                        int64_t* total_rows, int32_t* max_k);

/* Quantizes every row of descs_dev (device, a byte copy of a prepared
 * array, 8-byte aligned) in one launch, one workgroup per row. */
int sherry_quantize_act_batched(const sherry_quant_desc* descs_dev, int count,
                                int64_t total_rows, int32_t max_k, void* stream);

/* ---------------------------------------------------------------------- */
/* Online products (Eq. 2).                                                */
/* ---------------------------------------------------------------------- */

/* M = 1 product (decode).  w: device, packed layout of an n x k matrix,
 * 16-byte aligned.  x: device, int8 [k], 4-byte aligned.  x_scale: device,
 * fp32 [1].  w_scale: the per-tensor alpha.  y: device, fp32 [n], 4-byte
 * aligned.  acc: device, int32 [n] or NULL (then not written). */
int sherry_gemv(const uint8_t* w, const int8_t* x, const float* x_scale,
                float w_scale, float* y, int32_t* acc, int64_t n, int64_t k,
                void* stream);

/* Any-M product.  x: device, int8 [m][k] row-major, 16-byte aligned.
 * x_scale: device, fp32 [m].  y: device, fp32 [m][n]; acc: device, int32
 * [m][n] or NULL.  Other arguments as sherry_gemv.  Chooses the kernel by M
 * (see sherry_gemm_kernel_for). */
int sherry_gemm(const uint8_t* w, const int8_t* x, const float* x_scale,
                float w_scale, float* y, int32_t* acc, int64_t m, int64_t n,
                int64_t k, void* stream);

/* sherry_gemm with an explicit kernel (SHERRY_KERNEL_*); SHERRY_KERNEL_GEMV
 * requires m <= 4, SHERRY_KERNEL_ALUT m = 1 and k <= SHERRY_ALUT_MAX_K
 * (SHERRY_E_SHAPE otherwise).  Results are bit-identical across kernels. */
int sherry_gemm_ex(const uint8_t* w, const int8_t* x, const float* x_scale,
                   float w_scale, float* y, int32_t* acc, int64_t m,
                   int64_t n, int64_t k, int kernel, void* stream);

/* The kernel sherry_gemm picks for this shape, or -SHERRY_E_SHAPE for an
 * invalid shape: SHERRY_KERNEL_GEMV for m <= 4, SHERRY_KERNEL_SKINNY for
 * 5 <= m <= 8192, for k > n and for k >= 3072, else SHERRY_KERNEL_MFMA
 * (longer products with k <= 2048 and k <= n; thresholds measured on the
 * MI355X). */
int sherry_gemm_kernel_for(int64_t m, int64_t n, int64_t k);

/* sherry_gemm_ex with one weight scale per output channel: the footnote to
 * Eq. 2 scales column j of T by alpha_j, and Eq. 5 gives one alpha per
 * output channel.  w_scales: device, fp32 [n], 4-byte aligned (for example
 * the alpha that sherry_ternarize_pack writes).  y[i][j] = float(acc[i][j]) *
 * (x_scale[i] * w_scales[j]); the int32 acc is the same as sherry_gemm_ex's.
 * SHERRY_E_INVALID if w_scales is NULL. */
int sherry_gemm_channel(const uint8_t* w, const int8_t* x, const float* x_scale,
                        const float* w_scales, float* y, int32_t* acc, int64_t m,
                        int64_t n, int64_t k, int kernel, void* stream);

/* Per-group weight scales, group size 128 along k (the paper's default
 * granularity, Sec. 4.1; one scale per output channel and group).
 * w_group_scales: device, fp32 [n][ceil(k/128)] row-major, 4-byte aligned.
 * y[i][j] = x_scale[i] * sum_g float(acc_g[i][j]) * w_group_scales[j][g],
 * where acc_g is the exact int32 product over k in [128g, 128g + 128); the
 * sum runs in fp32 in ascending g within each part of the kernel's split of
 * k, and the parts are added in order (so y is within (G + 4) * 2^-24 of
 * x_scale * sum_g |acc_g * scale| of the exact value, G = ceil(k/128)).
 * acc, if not NULL, receives sum_g acc_g (the unscaled int32 product).
 * kernel: SHERRY_KERNEL_AUTO (GEMV for m <= 4, else register-decoded),
 * SHERRY_KERNEL_GEMV (m <= 4), SHERRY_KERNEL_GEMV_TOK (its limits, see
 * above; the partial sums are the exact per-group products of the lane's
 * row), SHERRY_KERNEL_SKINNY or SHERRY_KERNEL_MFMA (its 128 x 128 tile);
 * SHERRY_E_INVALID for SHERRY_KERNEL_ALUT and if w_group_scales is NULL. */
int sherry_gemm_group(const uint8_t* w, const int8_t* x, const float* x_scale,
                      const float* w_group_scales, float* y, int32_t* acc, int64_t m,
                      int64_t n, int64_t k, int kernel, void* stream);

/* ---------------------------------------------------------------------- */
/* Grouped M = 1 products: many independent GEMVs in one launch.           */
/* ---------------------------------------------------------------------- */

typedef struct sherry_gemv_desc {
  const uint8_t* w;      /* device, packed n x k, 16-byte aligned          */
  const int8_t* x;       /* device, int8 [k], 4-byte aligned               */
  const float* x_scale;  /* device, fp32 [1]                               */
  float* y;              /* device, fp32 [n]                               */
  int32_t* acc;          /* device, int32 [n] or NULL                      */
  const float* w_scales; /* device, fp32 [n] per-channel scales, or NULL   */
                         /* for the per-tensor w_scale                     */
  const float* w_group_scales; /* device, fp32 [n][ceil(k/128)] per-group  */
                         /* scales (as sherry_gemm_group), or NULL; at     */
                         /* most one of w_scales and w_group_scales is set */
  int32_t n, k;
  float w_scale;
  int32_t block_begin;   /* written by sherry_gemv_batched_prepare         */
} sherry_gemv_desc;

/* Host: validates descs[0..count) and fills each block_begin, the index of
 * the first workgroup of that product, and *total_blocks with their sum
 * (the number of workgroups depends on n and k through the library's work
 * split; descriptors only need to be prepared again if n or k change).
 * count >= 1. */
int sherry_gemv_batched_prepare(sherry_gemv_desc* descs, int count,
                                int64_t* total_blocks);

/* Runs every GEMV of descs_dev (device, a byte copy of an array accepted by
 * sherry_gemv_batched_prepare, 8-byte aligned) in one launch.  count and
 * total_blocks must be the values used with / returned by prepare; the
 * device descriptors cannot be re-validated here. */
int sherry_gemv_batched(const sherry_gemv_desc* descs_dev, int count,
                        int64_t total_blocks, void* stream);

/* ---------------------------------------------------------------------- */
/* Grouped products: many independent products (any m, e.g. the q, k and  */
/* v projections of one layer) in one launch: up to 4 tokens each on the   */
/* matrix-core GEMV (SHERRY_KERNEL_GEMV_TOK), up to 16 (without per-group */
/* scales) on a 16-token window kernel, else on the register-decoded kernel*/
/* (SHERRY_KERNEL_SKINNY), which runs token blocks of 32 when every        */
/* m <= 32 or a descriptor has per-group scales, else of 64.              */
/* ---------------------------------------------------------------------- */

/* Flag of a grouped launch value: some descriptor has per-group scales. */
#define SHERRY_LAUNCH_GROUPS (1 << 30)

typedef struct sherry_gemm_desc {
  const uint8_t* w;      /* device, packed n x k, 16-byte aligned          */
  const int8_t* x;       /* device, int8 [m][k], 16-byte aligned           */
  const float* x_scale;  /* device, fp32 [m]                               */
  float* y;              /* device, fp32 [m][n]                            */
  int32_t* acc;          /* device, int32 [m][n] or NULL                   */
  const float* w_scales; /* device, fp32 [n] per-channel scales, or NULL   */
  const float* w_group_scales; /* device, fp32 [n][ceil(k/128)] per-group  */
                         /* scales as in sherry_gemm_group, or NULL; not   */
                         /* with w_scales, and acc must then be NULL       */
  int32_t n, k, m;       /* 1 <= m <= SHERRY_MAX_M                         */
  float w_scale;
  int32_t block_begin;   /* written by prepare: the product's first block  */
  int32_t block_count;   /* written by prepare: its number of blocks       */
} sherry_gemm_desc;

/* Host: validates descs[0..count), fills each block_begin and block_count,
 * *total_blocks and *max_m, the launch value that selects the kernel and its
 * token blocks.  The blocks of the products are numbered in order of
 * decreasing k (ties in array order), whatever the order of the array: the
 * workgroups with the longest rows are dispatched first and the shorter ones
 * fill in behind them.  When every m <= 4 and every m * ceil(k/128) * 128 <= 32768, the
 * products run on the matrix-core GEMV (SHERRY_KERNEL_GEMV_TOK, any scales)
 * and *max_m is the largest m (1..4); else, when every m <= 16 and no
 * descriptor has per-group scales, on the 16-token window kernel (weights as
 * loaded, one int8 MFMA per 4-code chunk for 16 tokens x 64 rows) and *max_m
 * is the largest m, at least 5.  Otherwise they run on the register-decoded
 * kernel and *max_m is the largest m, at least 17, and at most 32 when a
 * descriptor carries per-group scales (their kernel runs 32-token blocks).
 * When a descriptor carries per-group scales, *max_m also has the bit
 * SHERRY_LAUNCH_GROUPS set (the kernels' per-group variants).  Pass it to
 * sherry_gemm_batched unchanged. */
int sherry_gemm_batched_prepare(sherry_gemm_desc* descs, int count,
                                int64_t* total_blocks, int32_t* max_m);

/* Runs every product of descs_dev (device, a byte copy of an array accepted
 * by sherry_gemm_batched_prepare, 8-byte aligned) in one launch; count,
 * total_blocks and max_m as returned by prepare. */
int sherry_gemm_batched(const sherry_gemm_desc* descs_dev, int count,
                        int64_t total_blocks, int32_t max_m, void* stream);

/* Grouped products of up to 16 tokens on lane-interleaved weights
 * (sherry_pack_il), per-tensor or per-channel scales: the 4-token GEMV
 * (every m <= 4 and m * ceil(k/128) * 128 <= 32768; launch value = the
 * largest m) or the 16-token window kernel (launch value = the largest m,
 * at least 5), each with one int8 MFMA per chunk slot and two activation
 * reads per unit.  _prepare validates as sherry_gemm_batched_prepare and
 * returns SHERRY_E_SHAPE for m > 16 and SHERRY_E_INVALID for per-group
 * scales.  Results bit-identical to sherry_gemm_batched on the tiled layout
 * of the same matrices (int32 sums exact, same epilogue). */
int sherry_gemm_il_batched_prepare(sherry_gemm_desc* descs, int count,
                                   int64_t* total_blocks, int32_t* max_m);
int sherry_gemm_il_batched(const sherry_gemm_desc* descs_dev, int count,
                           int64_t total_blocks, int32_t max_m, void* stream);

/* ---------------------------------------------------------------------- */
/* Fused quantization + M = 1 product: fp32 activations in, one launch.    */
/* Each workgroup quantizes the activation row (exactly as                 */
/* sherry_quantize_act) and runs the product of sherry_gemv on it, so the  */
/* results are bit-identical to sherry_quantize_act followed by            */
/* sherry_gemv, without the int8 round trip through memory and the second */
/* launch (the engine quantizes activations on the fly, Appendix A).       */
/* ---------------------------------------------------------------------- */

/* x: device, fp32 [k], 16-byte aligned, finite values, k <=
 * SHERRY_FUSED_MAX_K.  x_scale: device, fp32 [1] that receives the
 * activation scale (absmax / 127, 0 for an all-zero row), or NULL.  Other
 * arguments as sherry_gemv. */
int sherry_gemv_f32(const uint8_t* w, const float* x, float* x_scale,
                    float w_scale, float* y, int32_t* acc, int64_t n, int64_t k,
                    void* stream);

/* sherry_gemv_f32 with one weight scale per output channel (w_scales as in
 * sherry_gemm_channel). */
int sherry_gemv_f32_channel(const uint8_t* w, const float* x, float* x_scale,
                            const float* w_scales, float* y, int32_t* acc,
                            int64_t n, int64_t k, void* stream);

/* sherry_gemv_f32 with per-group weight scales (w_group_scales and the
 * result as in sherry_gemm_group). */
int sherry_gemv_f32_group(const uint8_t* w, const float* x, float* x_scale,
                          const float* w_group_scales, float* y, int32_t* acc,
                          int64_t n, int64_t k, void* stream);

typedef struct sherry_gemv_f32_desc {
  const uint8_t* w;      /* device, packed n x k, 16-byte aligned          */
  const float* x;        /* device, fp32 [k], 16-byte aligned              */
  float* x_scale;        /* device, fp32 [1] output, or NULL               */
  float* y;              /* device, fp32 [n]                               */
  int32_t* acc;          /* device, int32 [n] or NULL                      */
  const float* w_scales; /* device, fp32 [n] per-channel scales, or NULL   */
  const float* w_group_scales; /* per-group scales or NULL, as in          */
                         /* sherry_gemv_desc                               */
  int32_t n, k;          /* k <= SHERRY_FUSED_MAX_K                        */
  float w_scale;
  int32_t block_begin;   /* written by sherry_gemv_f32_batched_prepare     */
} sherry_gemv_f32_desc;

/* As sherry_gemv_batched_prepare / sherry_gemv_batched, for fused
 * descriptors: every product of the array runs in one launch. */
int sherry_gemv_f32_batched_prepare(sherry_gemv_f32_desc* descs, int count,
                                    int64_t* total_blocks);
int sherry_gemv_f32_batched(const sherry_gemv_f32_desc* descs_dev, int count,
                            int64_t total_blocks, void* stream);

/* The same fused products on lane-interleaved weights (sherry_pack_il): each
 * 4-code chunk slot of a lane is the B operand of one int8 MFMA over 16 rows
 * and 64 weights, whose activation operand serves the unit's four row
 * groups.  Results bit-identical to sherry_gemv_f32_batched on the tiled
 * layout of the same matrix.  Per-tensor or per-channel scales only:
 * _prepare returns SHERRY_E_INVALID for a descriptor with per-group scales,
 * otherwise it is sherry_gemv_f32_batched_prepare; pass its total_blocks. */
int sherry_gemv_f32_il_batched_prepare(sherry_gemv_f32_desc* descs, int count,
                                       int64_t* total_blocks);
int sherry_gemv_f32_il_batched(const sherry_gemv_f32_desc* descs_dev, int count,
                               int64_t total_blocks, void* stream);

/* ---------------------------------------------------------------------- */
/* Comparison layouts (Sec. 2.3): the "2-bit strategy" and the "1.67-bit   */
/* strategy" the paper sets against its 1.25-bit codes.  They hold any     */
/* ternary T and exist to measure bytes moved and time on the same GPU;    */
/* their products take int8 activations and one weight scale per tensor.  */
/*                                                                        */
/* 2-bit layout: one weight per 2 bits, value w+1; unit (r, c) = 64 rows x */
/* 64 weights = 1024 bytes at (r*Kp/64 + c)*1024, Kp = ceil(K/64)*64; row  */
/* i's 16 bytes at 16*i hold weight 64c + 16w + 4j + p (w, j, p in 0..3)   */
/* in byte 4w + p at bits [2j, 2j+2); padding is weight 0.                */
/*                                                                        */
/* 1.67-bit layout: three weights per 5-bit code, code = (t0+1) + 3(t1+1)  */
/* + 9(t2+1) for the block t0, t1, t2 of weights 3b, 3b+1, 3b+2 (codes     */
/* 27..31 unused); T is extended with zero weights to Np = ceil(N/64)*64   */
/* rows and Kp = ceil(K/96)*96 columns; unit (r, c) = 64 rows x 96 weights */
/* = 1280 bytes at (r*Kp/96 + c)*1280, laid out as a 5-bit unit: row i's   */
/* 160-bit stream holds code j (weights 96c + 3j .. + 2) at stream bits    */
/* [5j, 5j+5), stream bits 0..127 in bytes 16*i.., 128..159 in            */
/* 1024 + 4*i...                                                          */
/* ---------------------------------------------------------------------- */

size_t sherry_packed2_bytes(int64_t n, int64_t k);

/* Packs any ternary T (host, int8 [n][k] in {-1,0,1}); SHERRY_E_INVALID for
 * another value, its flat index in *bad_index when not NULL. */
int sherry_pack2(const int8_t* t, int64_t n, int64_t k, uint8_t* out,
                 size_t out_bytes, int64_t* bad_index);

/* M = 1 product on the 2-bit layout; arguments as sherry_gemv. */
int sherry_gemv2(const uint8_t* w2, const int8_t* x, const float* x_scale,
                 float w_scale, float* y, int32_t* acc, int64_t n, int64_t k,
                 void* stream);

/* Bytes of the 1.67-bit layout of an n x k matrix (any k >= 1), or 0 if
 * n < 1, k < 1, n > SHERRY_MAX_N or k > SHERRY_MAX_K. */
size_t sherry_packed3_bytes(int64_t n, int64_t k);

/* Packs any ternary T (host, int8 [n][k] in {-1,0,1}) into the 1.67-bit
 * layout (host buffer of at least sherry_packed3_bytes(n, k) bytes, every
 * byte written); SHERRY_E_INVALID for another value, its flat index in
 * *bad_index when not NULL. */
int sherry_pack3(const int8_t* t, int64_t n, int64_t k, uint8_t* out,
                 size_t out_bytes, int64_t* bad_index);

/* Inverse of sherry_pack3 (host); SHERRY_E_INVALID if a code of the first n
 * rows and k weights is one of the unused codes 27..31. */
int sherry_unpack3(const uint8_t* packed, size_t packed_bytes, int64_t n,
                   int64_t k, int8_t* t_out);

/* M = 1 product on the 1.67-bit layout; arguments as sherry_gemv (k % 4 ==
 * 0 for the int8 activation words). */
int sherry_gemv3(const uint8_t* w3, const int8_t* x, const float* x_scale,
                 float w_scale, float* y, int32_t* acc, int64_t n, int64_t k,
                 void* stream);

/* Grouped M = 1 products on the 2-bit (gemv2) or 1.67-bit (gemv3) layout:
 * as sherry_gemv_batched_prepare / sherry_gemv_batched, with descriptors
 * whose w points to that layout; w_scales and w_group_scales must be NULL
 * (SHERRY_E_INVALID otherwise). */
int sherry_gemv2_batched_prepare(sherry_gemv_desc* descs, int count,
                                 int64_t* total_blocks);
int sherry_gemv2_batched(const sherry_gemv_desc* descs_dev, int count,
                         int64_t total_blocks, void* stream);
int sherry_gemv3_batched_prepare(sherry_gemv_desc* descs, int count,
                                 int64_t* total_blocks);
int sherry_gemv3_batched(const sherry_gemv_desc* descs_dev, int count,
                         int64_t total_blocks, void* stream);

/* ---------------------------------------------------------------------- */
/* Diagnostics.                                                            */
/* ---------------------------------------------------------------------- */

/* Streaming-read ceiling probe: reads `bytes` (multiple of 16, src 16-byte
 * aligned) with the loads the products use for their packed weights (128-bit
 * buffer loads, non-temporal hint) and writes one XOR checksum word per
 * workgroup to sink (device, uint32 [sherry_stream_read_groups(bytes)]). */
int sherry_stream_read(const void* src, size_t bytes, uint32_t* sink,
                       void* stream);
int64_t sherry_stream_read_groups(size_t bytes);

#ifdef __cplusplus
}
#endif

#endif /* SHERRY_H_ */
