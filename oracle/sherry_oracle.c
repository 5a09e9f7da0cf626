/*
 * sherry_oracle.c -- plain, slow, obviously-correct CPU oracle for the Sherry
 * 3:4 sparse ternary product (arXiv 2601.07892).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library may include, link,
 * load or call this file.  Only the tests, the smoke check and the CPU-baseline
 * leg of the benchmark use it.  It shares no code, header, table or constant
 * with the HIP path; the two meet only at the bytes of the packed format and
 * at the numbers they compute.
 *
 * What it computes, and the passage each part follows:
 *
 *  (i)   code table    -- Sec. 3.1, "sweet spot" point (3): a 4-weight block
 *                         with exactly one zero and three signs has
 *                         C(4,3)*2^3 = 32 states, one per 5-bit code.  The
 *                         assignment of bits is this project's reading: low 2
 *                         bits = position of the zero inside the block, bit
 *                         2+i = sign of the i-th non-zero in ascending
 *                         position (1 means -1).  Built by enumerating all 81
 *                         ternary 4-tuples.
 *  (ii)  pack/unpack   -- Appendix A (offline packing phase): each 4-block is
 *                         stored as one 5-bit code in a word-aligned stream.
 *                         The stream layout is this project's own (the paper
 *                         gives none); it is written out bit by bit below.
 *  (iii) act. quant.   -- not in the paper (weight-only, Limitations) yet the
 *                         engine accumulates in integers (Appendix A, online
 *                         phase): int8 per-token absmax/127, fp32 decisions.
 *  (iv)  product       -- Eq. 2, Y = X T alpha, with T in {-1,0,1} satisfying
 *                         the 3:4 constraint of Eq. 3.  Plain dense integer
 *                         triple loop on the UNPACKED T; never reads a code.
 *  (v)   epilogue      -- Eq. 2 scaling, y = acc * sx * sw, in fp64; also
 *                         with one sw per output channel ([T alpha]_ij =
 *                         T_ij alpha_j, the footnote to Eq. 2).
 *  (vi)  ternarizer    -- Eq. 4 (Sparse-AbsMean) and Eq. 5 (alpha), with a
 *                         per-tensor alpha, or one alpha per output channel
 *                         as Eq. 5 states it.
 *  (vii) 2-bit codec   -- the "2-bit strategy" of Sec. 2.3 (one ternary
 *                         weight per 2 bits), used only as a bytes-moved
 *                         comparison; layout is this project's own.
 *  (viii) 1.67-bit codec -- the "1.67-bit strategy" of Sec. 2.3: three
 *                         ternary weights per 5-bit code, 3^3 = 27 of the 32
 *                         codes used.  The digit order is this project's
 *                         reading: code = (t0+1) + 3(t1+1) + 9(t2+1) for the
 *                         weights t0, t1, t2 of a block in ascending K.
 *                         Built by enumerating the 27 triples.  Comparison
 *                         layout only.
 *
 *  (ix)  lane-interleaved layout -- this project's own placement of the codes
 *                         of (ii) for the int8 matrix-core products: same
 *                         units, containers and stream bits, another
 *                         assignment of a unit's (row, block) pairs to
 *                         (container, code) slots.  Written out below.
 *
 *  Parity unpinned: the bit assignment inside a code (i) and the placement of
 *  the codes in the stream (ii).  The paper prints no packed example, so the
 *  tests pin them only to the written reading (a hand-written code table and
 *  hand-derived byte fixtures under tests/golden), not to the paper.
 *
 * Build: gcc -O2 -std=c11 -fPIC -shared -ffp-contract=off -pthread.
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* ------------------------------------------------------------------------ */
/* (i) code table by enumeration                                            */
/* ------------------------------------------------------------------------ */

static int8_t g_table[32][4];
static int g_table_ready = 0;

/* Fills table[c][p] = weight at block position p for code c.  Returns the
 * number of ternary 4-tuples accepted (must be 32; 81 are enumerated). */
int oracle_code_table(int8_t table[32][4]) {
  int accepted = 0;
  int filled[32];
  for (int c = 0; c < 32; ++c) filled[c] = 0;
  const int vals[3] = {-1, 0, 1};
  for (int a = 0; a < 3; ++a)
    for (int b = 0; b < 3; ++b)
      for (int d = 0; d < 3; ++d)
        for (int e = 0; e < 3; ++e) {
          int w[4] = {vals[a], vals[b], vals[d], vals[e]};
          int zeros = 0, zpos = -1;
          for (int p = 0; p < 4; ++p)
            if (w[p] == 0) { ++zeros; zpos = p; }
          if (zeros != 1) continue; /* violates the 3:4 constraint (Eq. 3) */
          /* signs of the three non-zeros, in ascending position */
          int code = zpos, i = 0;
          for (int p = 0; p < 4; ++p) {
            if (p == zpos) continue;
            if (w[p] < 0) code += 1 << (2 + i);
            ++i;
          }
          if (filled[code]) return -1; /* two tuples on one code: broken */
          filled[code] = 1;
          for (int p = 0; p < 4; ++p) table[code][p] = (int8_t)w[p];
          ++accepted;
        }
  return accepted;
}

static void ensure_table(void) {
  if (!g_table_ready) {
    oracle_code_table(g_table);
    g_table_ready = 1;
  }
}

/* Code of one block by searching the table; -1 if the block is not 3:4. */
int oracle_encode_block(const int8_t w[4]) {
  ensure_table();
  for (int c = 0; c < 32; ++c) {
    if (g_table[c][0] == w[0] && g_table[c][1] == w[1] &&
        g_table[c][2] == w[2] && g_table[c][3] == w[3])
      return c;
  }
  return -1;
}

void oracle_decode_code(int c, int8_t w[4]) {
  ensure_table();
  for (int p = 0; p < 4; ++p) w[p] = g_table[c & 31][p];
}

/* ------------------------------------------------------------------------ */
/* (ii) the 5-bit tiled layout, bit by bit                                  */
/*                                                                          */
/* Rows are padded to Np = ceil(N/64)*64 and the reduction dimension to      */
/* Kp = ceil(K/128)*128; padding codes are all-zero bits.  The matrix is a   */
/* grid of units of 64 rows x 128 weights (1280 bytes), unit (r, c) at byte  */
/* (r*C + c)*1280 with C = Kp/128.  Inside a unit, row i (0..63) holds one   */
/* container of 32 consecutive codes for weights 128*c .. 128*c+127: a       */
/* 160-bit little-endian stream, code j at stream bits [5j, 5j+5) (code bit  */
/* q at stream bit 5j+q).  Stream bits 0..127 go to the head bytes at        */
/* 16*i + (0..15); stream bits 128..159 to the tail bytes at 1024 + 4*i +    */
/* (0..3).  Inside a byte, stream bit 8*p + t is bit t (LSB first).          */
/* ------------------------------------------------------------------------ */

static int64_t ceil_to(int64_t v, int64_t m) { return (v + m - 1) / m * m; }

int64_t oracle_packed_bytes(int64_t n, int64_t k) {
  if (n < 1 || k < 1 || k % 4 != 0) return 0;
  return ceil_to(n, 64) * ceil_to(k, 128) * 5 / 32;
}

/* Byte offset and bit inside it for stream bit sp of the container of row n
 * and container column c, in a matrix with C container columns. */
static void stream_bit_addr(int64_t n, int64_t c, int sp, int64_t C,
                            int64_t* byte, int* bit) {
  int64_t r = n / 64;
  int i = (int)(n % 64);
  int64_t unit = (r * C + c) * 1280;
  if (sp < 128) {
    *byte = unit + 16 * i + sp / 8;
    *bit = sp % 8;
  } else {
    *byte = unit + 1024 + 4 * i + (sp - 128) / 8;
    *bit = (sp - 128) % 8;
  }
}

/* Packs T (N x K, row-major, values in {-1,0,1}) into out, which must hold
 * oracle_packed_bytes(n, k) bytes.  Returns 0, or -(b+1) where b is the flat
 * index (n*K/4 + block) of the first block that is not 3:4. */
int64_t oracle_pack(const int8_t* t, int64_t n, int64_t k, uint8_t* out) {
  int64_t bytes = oracle_packed_bytes(n, k);
  if (bytes == 0) return -((int64_t)1 << 62);
  memset(out, 0, (size_t)bytes);
  int64_t C = ceil_to(k, 128) / 128;
  int64_t nb = k / 4;
  for (int64_t row = 0; row < n; ++row) {
    for (int64_t b = 0; b < nb; ++b) {
      int code = oracle_encode_block(t + row * k + 4 * b);
      if (code < 0) return -(row * nb + b + 1);
      int64_t kk = 4 * b;            /* first weight of the block      */
      int64_t c = kk / 128;          /* container column               */
      int j = (int)((kk % 128) / 4); /* code inside the container      */
      for (int q = 0; q < 5; ++q) {
        int64_t byte;
        int bit;
        stream_bit_addr(row, c, 5 * j + q, C, &byte, &bit);
        if ((code >> q) & 1) out[byte] |= (uint8_t)(1u << bit);
      }
    }
  }
  return 0;
}

/* Inverse of oracle_pack for the first n rows and k weights. */
int oracle_unpack(const uint8_t* p, int64_t n, int64_t k, int8_t* t) {
  if (oracle_packed_bytes(n, k) == 0) return -1;
  int64_t C = ceil_to(k, 128) / 128;
  for (int64_t row = 0; row < n; ++row) {
    for (int64_t b = 0; b < k / 4; ++b) {
      int64_t kk = 4 * b;
      int64_t c = kk / 128;
      int j = (int)((kk % 128) / 4);
      int code = 0;
      for (int q = 0; q < 5; ++q) {
        int64_t byte;
        int bit;
        stream_bit_addr(row, c, 5 * j + q, C, &byte, &bit);
        code |= ((p[byte] >> bit) & 1) << q;
      }
      oracle_decode_code(code, t + row * k + kk);
    }
  }
  return 0;
}

/* ------------------------------------------------------------------------ */
/* (iii) activation quantization: int8 per token, absmax/127                */
/* Decisions in fp32 (IEEE division, round-half-to-even), as the kernel.    */
/* ------------------------------------------------------------------------ */

void oracle_quantize_act(const float* x, int64_t m, int64_t k, int8_t* q,
                         float* sx) {
  for (int64_t r = 0; r < m; ++r) {
    const float* xr = x + r * k;
    float amax = 0.0f;
    for (int64_t i = 0; i < k; ++i) {
      float a = fabsf(xr[i]);
      if (a > amax) amax = a;
    }
    if (amax == 0.0f) {
      sx[r] = 0.0f;
      for (int64_t i = 0; i < k; ++i) q[r * k + i] = 0;
      continue;
    }
    volatile float s = amax / 127.0f; /* volatile: keep it an fp32 value */
    sx[r] = s;
    for (int64_t i = 0; i < k; ++i) {
      volatile float v = xr[i] / s;
      float rv = rintf(v); /* default rounding mode: to nearest, ties even */
      if (rv > 127.0f) rv = 127.0f;
      if (rv < -127.0f) rv = -127.0f;
      q[r * k + i] = (int8_t)rv;
    }
  }
}

/* ------------------------------------------------------------------------ */
/* (iv) the product of Eq. 2 on the unpacked T, plain triple loop           */
/* acc[m][n] = sum_k x[m][k] * t[n][k]                                      */
/* ------------------------------------------------------------------------ */

typedef struct {
  const int8_t* x;
  const int8_t* t;
  int32_t* acc;
  int64_t m, n, k, n0, n1;
} gemm_job;

static void* gemm_rows(void* arg) {
  gemm_job* j = (gemm_job*)arg;
  for (int64_t mm = 0; mm < j->m; ++mm) {
    for (int64_t nn = j->n0; nn < j->n1; ++nn) {
      int64_t sum = 0;
      for (int64_t kk = 0; kk < j->k; ++kk)
        sum += (int64_t)j->x[mm * j->k + kk] * (int64_t)j->t[nn * j->k + kk];
      j->acc[mm * j->n + nn] = (int32_t)sum;
    }
  }
  return 0;
}

/* threads <= 1 runs on the calling thread; otherwise output rows n are split
 * into `threads` contiguous ranges. */
void oracle_gemm_i32(const int8_t* x, const int8_t* t, int64_t m, int64_t n,
                     int64_t k, int32_t* acc, int threads) {
  if (threads <= 1 || n < threads) {
    gemm_job j = {x, t, acc, m, n, k, 0, n};
    gemm_rows(&j);
    return;
  }
  pthread_t* th = (pthread_t*)malloc(sizeof(pthread_t) * (size_t)threads);
  gemm_job* jobs = (gemm_job*)malloc(sizeof(gemm_job) * (size_t)threads);
  for (int i = 0; i < threads; ++i) {
    gemm_job j = {x, t, acc, m, n, k, n * i / threads, n * (i + 1) / threads};
    jobs[i] = j;
    pthread_create(&th[i], 0, gemm_rows, &jobs[i]);
  }
  for (int i = 0; i < threads; ++i) pthread_join(th[i], 0);
  free(th);
  free(jobs);
}

/* Single output element, for sampled checks at full size. */
int32_t oracle_dot_i32(const int8_t* x_row, const int8_t* t_row, int64_t k) {
  int64_t sum = 0;
  for (int64_t kk = 0; kk < k; ++kk) sum += (int64_t)x_row[kk] * t_row[kk];
  return (int32_t)sum;
}

/* ------------------------------------------------------------------------ */
/* (v) epilogue in fp64: y = acc * sx[m] * sw                               */
/* ------------------------------------------------------------------------ */

void oracle_epilogue(const int32_t* acc, const float* sx, float sw, int64_t m,
                     int64_t n, double* y) {
  for (int64_t mm = 0; mm < m; ++mm)
    for (int64_t nn = 0; nn < n; ++nn)
      y[mm * n + nn] = (double)acc[mm * n + nn] * (double)sx[mm] * (double)sw;
}

/* Per-output-channel scales: y = acc * sx[m] * sw[n]. */
void oracle_epilogue_rows(const int32_t* acc, const float* sx, const float* sw,
                          int64_t m, int64_t n, double* y) {
  for (int64_t mm = 0; mm < m; ++mm)
    for (int64_t nn = 0; nn < n; ++nn)
      y[mm * n + nn] = (double)acc[mm * n + nn] * (double)sx[mm] * (double)sw[nn];
}

/* ------------------------------------------------------------------------ */
/* (vi) Sparse-AbsMean ternarizer, Eq. 4 and Eq. 5 (per-tensor alpha)       */
/* Ties for the smallest |W| go to the lowest position; a kept weight equal */
/* to zero gets +1 so that every block keeps exactly one zero.              */
/* ------------------------------------------------------------------------ */

double oracle_ternarize(const float* w, int64_t n, int64_t k, int8_t* t) {
  double kept_abs = 0.0;
  int64_t kept = 0;
  for (int64_t row = 0; row < n; ++row) {
    for (int64_t b = 0; b < k / 4; ++b) {
      const float* wb = w + row * k + 4 * b;
      int amin = 0;
      for (int p = 1; p < 4; ++p)
        if (fabs((double)wb[p]) < fabs((double)wb[amin])) amin = p;
      for (int p = 0; p < 4; ++p) {
        int8_t v;
        if (p == amin) {
          v = 0;
        } else {
          v = (wb[p] < 0.0f) ? -1 : 1;
          kept_abs += fabs((double)wb[p]);
          ++kept;
        }
        t[row * k + 4 * b + p] = v;
      }
    }
  }
  return kept ? kept_abs / (double)kept : 0.0;
}

/* Eq. 5 as the paper states it: one alpha per output channel (row of T),
 * the mean |W| over that row's kept weights, summed in fp64 in ascending K
 * order.  T is the same as oracle_ternarize's. */
void oracle_ternarize_rows(const float* w, int64_t n, int64_t k, int8_t* t,
                           double* alpha) {
  for (int64_t row = 0; row < n; ++row) {
    double kept_abs = 0.0;
    int64_t kept = 0;
    for (int64_t b = 0; b < k / 4; ++b) {
      const float* wb = w + row * k + 4 * b;
      int amin = 0;
      for (int p = 1; p < 4; ++p)
        if (fabs((double)wb[p]) < fabs((double)wb[amin])) amin = p;
      for (int p = 0; p < 4; ++p) {
        int8_t v = 0;
        if (p != amin) {
          v = (wb[p] < 0.0f) ? -1 : 1;
          kept_abs += fabs((double)wb[p]);
          ++kept;
        }
        t[row * k + 4 * b + p] = v;
      }
    }
    alpha[row] = kept ? kept_abs / (double)kept : 0.0;
  }
}

/* ------------------------------------------------------------------------ */
/* (vii) 2-bit layout: value w+1 in {0,1,2}, bit by bit                     */
/* Rows padded to ceil(N/64)*64, reduction dim to ceil(K/64)*64 (padding     */
/* value 1, i.e. weight 0).  Unit (r, c) of 64 rows x 64 weights is 1024     */
/* bytes at (r*C + c)*1024 with C = Kp/64; row i holds the 16 bytes at       */
/* 16*i.  Weight 64*c + u, u = 16*w + 4*j + p (w, j, p in 0..3), sits in     */
/* byte 4*w + p of those 16, at bits [2j, 2j+2): byte p of 32-bit word w     */
/* gathers the 2-bit fields of weights 16w + p, 16w + 4 + p, 16w + 8 + p and */
/* 16w + 12 + p.                                                             */
/* ------------------------------------------------------------------------ */

int64_t oracle_packed2_bytes(int64_t n, int64_t k) {
  if (n < 1 || k < 1 || k % 4 != 0) return 0;
  return ceil_to(n, 64) * ceil_to(k, 64) / 4;
}

static int64_t two_bit_byte(int64_t row, int64_t kk, int q, int64_t C, int* bit) {
  int64_t r = row / 64, c = kk / 64;
  int i = (int)(row % 64);
  int u = (int)(kk % 64);
  int w = u / 16, j = (u % 16) / 4, p = u % 4;
  *bit = 2 * j + q;
  return (r * C + c) * 1024 + 16 * i + 4 * w + p;
}

int64_t oracle_pack2(const int8_t* t, int64_t n, int64_t k, uint8_t* out) {
  int64_t bytes = oracle_packed2_bytes(n, k);
  if (bytes == 0) return -((int64_t)1 << 62);
  int64_t C = ceil_to(k, 64) / 64;
  int64_t np = ceil_to(n, 64), kp = ceil_to(k, 64);
  memset(out, 0, (size_t)bytes);
  for (int64_t row = 0; row < np; ++row) {
    for (int64_t kk = 0; kk < kp; ++kk) {
      int v = 1; /* weight 0 */
      if (row < n && kk < k) {
        int8_t w = t[row * k + kk];
        if (w < -1 || w > 1) return -(row * k + kk + 1);
        v = w + 1;
      }
      for (int q = 0; q < 2; ++q) {
        int bit;
        int64_t byte = two_bit_byte(row, kk, q, C, &bit);
        if ((v >> q) & 1) out[byte] |= (uint8_t)(1u << bit);
      }
    }
  }
  return 0;
}

int oracle_unpack2(const uint8_t* pk, int64_t n, int64_t k, int8_t* t) {
  if (oracle_packed2_bytes(n, k) == 0) return -1;
  int64_t C = ceil_to(k, 64) / 64;
  for (int64_t row = 0; row < n; ++row) {
    for (int64_t kk = 0; kk < k; ++kk) {
      int v = 0;
      for (int q = 0; q < 2; ++q) {
        int bit;
        int64_t byte = two_bit_byte(row, kk, q, C, &bit);
        v |= ((pk[byte] >> bit) & 1) << q;
      }
      if (v > 2) return -2;
      t[row * k + kk] = (int8_t)(v - 1);
    }
  }
  return 0;
}

/* ------------------------------------------------------------------------ */
/* (viii) 1.67-bit layout: three weights per 5-bit code, bit by bit         */
/*                                                                          */
/* The matrix is extended with zero weights to Np = ceil(N/64)*64 rows and   */
/* Kp = ceil(K/96)*96 columns.  Block b of a row is weights 3b, 3b+1, 3b+2;  */
/* its code is (t0+1) + 3*(t1+1) + 9*(t2+1) (0..26; an all-zero block is     */
/* 13).  Unit (r, c) of 64 rows x 96 weights (32 codes per row) is 1280      */
/* bytes at (r*C + c)*1280 with C = Kp/96; inside it the codes sit exactly   */
/* as in the 5-bit layout (ii): row i's 160-bit stream holds code j of the   */
/* unit (weights 96c + 3j .. 96c + 3j + 2) at stream bits [5j, 5j+5), stream */
/* bits 0..127 in bytes 16*i + (0..15), bits 128..159 in 1024 + 4*i + (0..3).*/
/* ------------------------------------------------------------------------ */

static int8_t g_table3[27][3];
static int g_table3_ready = 0;

/* Fills table[code] = (t0, t1, t2) by enumerating every ternary triple;
 * returns the number of codes used (27). */
int oracle_code3_table(int8_t table[27][3]) {
  int used = 0;
  for (int t2 = -1; t2 <= 1; ++t2)
    for (int t1 = -1; t1 <= 1; ++t1)
      for (int t0 = -1; t0 <= 1; ++t0) {
        int code = (t0 + 1) + 3 * (t1 + 1) + 9 * (t2 + 1);
        table[code][0] = (int8_t)t0;
        table[code][1] = (int8_t)t1;
        table[code][2] = (int8_t)t2;
        ++used;
      }
  return used;
}

static void ensure_table3(void) {
  if (!g_table3_ready) {
    oracle_code3_table(g_table3);
    g_table3_ready = 1;
  }
}

/* Code of a block of three weights, or -1 if a weight is not in {-1,0,1}. */
int oracle_encode3(const int8_t w[3]) {
  ensure_table3();
  for (int c = 0; c < 27; ++c)
    if (g_table3[c][0] == w[0] && g_table3[c][1] == w[1] && g_table3[c][2] == w[2]) return c;
  return -1;
}

int64_t oracle_packed3_bytes(int64_t n, int64_t k) {
  if (n < 1 || k < 1) return 0;
  return ceil_to(n, 64) * (ceil_to(k, 96) / 96) * 20;
}

static void stream3_bit_addr(int64_t row, int64_t c, int sp, int64_t C, int64_t* byte,
                             int* bit) {
  int64_t r = row / 64;
  int i = (int)(row % 64);
  int64_t unit = (r * C + c) * 1280;
  if (sp < 128) {
    *byte = unit + 16 * i + sp / 8;
    *bit = sp % 8;
  } else {
    *byte = unit + 1024 + 4 * i + (sp - 128) / 8;
    *bit = (sp - 128) % 8;
  }
}

/* Packs T (N x K, values in {-1,0,1}); returns 0, or -(e+1) for the flat
 * index e (n*K + k) of the first weight outside {-1,0,1}. */
int64_t oracle_pack3(const int8_t* t, int64_t n, int64_t k, uint8_t* out) {
  int64_t bytes = oracle_packed3_bytes(n, k);
  if (bytes == 0) return -((int64_t)1 << 62);
  for (int64_t e = 0; e < n * k; ++e)
    if (t[e] < -1 || t[e] > 1) return -(e + 1);
  memset(out, 0, (size_t)bytes);
  int64_t np = ceil_to(n, 64), kp = ceil_to(k, 96), C = kp / 96;
  for (int64_t row = 0; row < np; ++row) {
    for (int64_t b = 0; b < kp / 3; ++b) {
      int8_t w[3];
      for (int q = 0; q < 3; ++q) {
        int64_t kk = 3 * b + q;
        w[q] = (row < n && kk < k) ? t[row * k + kk] : 0;
      }
      int code = oracle_encode3(w);
      int64_t c = (3 * b) / 96;
      int j = (int)(b % 32);
      for (int q = 0; q < 5; ++q) {
        int64_t byte;
        int bit;
        stream3_bit_addr(row, c, 5 * j + q, C, &byte, &bit);
        if ((code >> q) & 1) out[byte] |= (uint8_t)(1u << bit);
      }
    }
  }
  return 0;
}

/* Inverse of oracle_pack3 for the first n rows and k weights; returns -2 if
 * a code read there is one of the five unused ones (27..31). */
int oracle_unpack3(const uint8_t* p, int64_t n, int64_t k, int8_t* t) {
  if (oracle_packed3_bytes(n, k) == 0) return -1;
  ensure_table3();
  int64_t C = ceil_to(k, 96) / 96;
  for (int64_t row = 0; row < n; ++row) {
    for (int64_t b = 0; b < (k + 2) / 3; ++b) {
      int64_t c = (3 * b) / 96;
      int j = (int)(b % 32);
      int code = 0;
      for (int q = 0; q < 5; ++q) {
        int64_t byte;
        int bit;
        stream3_bit_addr(row, c, 5 * j + q, C, &byte, &bit);
        code |= ((p[byte] >> bit) & 1) << q;
      }
      if (code > 26) return -2;
      for (int q = 0; q < 3; ++q)
        if (3 * b + q < k) t[row * k + 3 * b + q] = g_table3[code][q];
    }
  }
  return 0;
}

/* ------------------------------------------------------------------------ */
/* (ix) lane-interleaved layout                                             */
/*                                                                          */
/* Units, containers (16-byte head at 16*l, 4-byte tail at 1024 + 4*l for    */
/* container l = 0..63) and the 160-bit stream of a container are those of   */
/* (ii).  Only the slot of each code differs: row i of a unit, written       */
/* i = 16g + t (g = 0..3, t = 0..15), and block b of the unit (weights        */
/* 4b..4b+3 of its 128), written b = 16p + 4h + c (p = 0..1, h = 0..3,        */
/* c = 0..3), go to container 16h + t as code 4(2g + p) + c.                  */
/* ------------------------------------------------------------------------ */

static void il_slot(int i, int b, int* container, int* code) {
  int g = i / 16, t = i % 16;
  int p = b / 16, h = (b / 4) % 4, c = b % 4;
  *container = 16 * h + t;
  *code = 4 * (2 * g + p) + c;
}

/* Byte and bit of stream bit sp of container l of unit (r, c). */
static void il_bit_addr(int64_t r, int64_t c, int l, int sp, int64_t C, int64_t* byte,
                        int* bit) {
  int64_t unit = (r * C + c) * 1280;
  if (sp < 128) {
    *byte = unit + 16 * l + sp / 8;
    *bit = sp % 8;
  } else {
    *byte = unit + 1024 + 4 * l + (sp - 128) / 8;
    *bit = (sp - 128) % 8;
  }
}

/* As oracle_pack, in the lane-interleaved layout. */
int64_t oracle_pack_il(const int8_t* t, int64_t n, int64_t k, uint8_t* out) {
  int64_t bytes = oracle_packed_bytes(n, k);
  if (bytes == 0) return -((int64_t)1 << 62);
  memset(out, 0, (size_t)bytes);
  int64_t C = ceil_to(k, 128) / 128;
  int64_t nb = k / 4;
  for (int64_t row = 0; row < n; ++row) {
    for (int64_t b = 0; b < nb; ++b) {
      int code = oracle_encode_block(t + row * k + 4 * b);
      if (code < 0) return -(row * nb + b + 1);
      int l, j;
      il_slot((int)(row % 64), (int)(b % 32), &l, &j);
      for (int q = 0; q < 5; ++q) {
        int64_t byte;
        int bit;
        il_bit_addr(row / 64, b / 32, l, 5 * j + q, C, &byte, &bit);
        if ((code >> q) & 1) out[byte] |= (uint8_t)(1u << bit);
      }
    }
  }
  return 0;
}

/* Inverse of oracle_pack_il for the first n rows and k weights. */
int oracle_unpack_il(const uint8_t* p, int64_t n, int64_t k, int8_t* t) {
  if (oracle_packed_bytes(n, k) == 0) return -1;
  int64_t C = ceil_to(k, 128) / 128;
  for (int64_t row = 0; row < n; ++row) {
    for (int64_t b = 0; b < k / 4; ++b) {
      int l, j;
      il_slot((int)(row % 64), (int)(b % 32), &l, &j);
      int code = 0;
      for (int q = 0; q < 5; ++q) {
        int64_t byte;
        int bit;
        il_bit_addr(row / 64, b / 32, l, 5 * j + q, C, &byte, &bit);
        code |= ((p[byte] >> bit) & 1) << q;
      }
      oracle_decode_code(code, t + row * k + 4 * b);
    }
  }
  return 0;
}
