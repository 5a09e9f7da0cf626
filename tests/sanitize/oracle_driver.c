/* Exercises every entry point of the C oracle on ragged shapes, built with
 * AddressSanitizer and UndefinedBehaviorSanitizer on the host (CPU only).
 * Exit status 0 when every round trip and closed form holds. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

int oracle_code_table(int8_t table[32][4]);
int oracle_encode_block(const int8_t w[4]);
void oracle_decode_code(int c, int8_t w[4]);
int64_t oracle_packed_bytes(int64_t n, int64_t k);
int64_t oracle_pack(const int8_t* t, int64_t n, int64_t k, uint8_t* out);
int oracle_unpack(const uint8_t* p, int64_t n, int64_t k, int8_t* t);
void oracle_quantize_act(const float* x, int64_t m, int64_t k, int8_t* q, float* sx);
void oracle_gemm_i32(const int8_t* x, const int8_t* t, int64_t m, int64_t n, int64_t k,
                     int32_t* acc, int threads);
int32_t oracle_dot_i32(const int8_t* x_row, const int8_t* t_row, int64_t k);
void oracle_epilogue(const int32_t* acc, const float* sx, float sw, int64_t m, int64_t n,
                     double* y);
void oracle_epilogue_rows(const int32_t* acc, const float* sx, const float* sw, int64_t m,
                          int64_t n, double* y);
double oracle_ternarize(const float* w, int64_t n, int64_t k, int8_t* t);
void oracle_ternarize_rows(const float* w, int64_t n, int64_t k, int8_t* t, double* alpha);
int64_t oracle_packed2_bytes(int64_t n, int64_t k);
int64_t oracle_pack2(const int8_t* t, int64_t n, int64_t k, uint8_t* out);
int oracle_unpack2(const uint8_t* pk, int64_t n, int64_t k, int8_t* t);

static uint64_t g_state = 0x9E3779B97F4A7C15ull;
static uint64_t next_u64(void) { /* SplitMix64 */
  uint64_t z = (g_state += 0x9E3779B97F4A7C15ull);
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

#define CHECK(c)                                              \
  do {                                                        \
    if (!(c)) {                                               \
      fprintf(stderr, "check failed: %s (line %d)\n", #c, __LINE__); \
      return 1;                                               \
    }                                                         \
  } while (0)

static int one_shape(int64_t m, int64_t n, int64_t k) {
  int8_t* t = malloc((size_t)(n * k));
  int8_t* t2 = malloc((size_t)(n * k));
  int8_t table[32][4];
  CHECK(oracle_code_table(table) == 32);
  for (int64_t i = 0; i < n * k / 4; ++i) memcpy(t + 4 * i, table[next_u64() % 32], 4);
  const int64_t nb = oracle_packed_bytes(n, k);
  uint8_t* p = malloc((size_t)nb);
  CHECK(oracle_pack(t, n, k, p) == 0);
  CHECK(oracle_unpack(p, n, k, t2) == 0);
  CHECK(memcmp(t, t2, (size_t)(n * k)) == 0);
  const int64_t nb2 = oracle_packed2_bytes(n, k);
  uint8_t* p2 = malloc((size_t)nb2);
  CHECK(oracle_pack2(t, n, k, p2) == 0);
  CHECK(oracle_unpack2(p2, n, k, t2) == 0);
  CHECK(memcmp(t, t2, (size_t)(n * k)) == 0);

  float* x = malloc(sizeof(float) * (size_t)(m * k));
  for (int64_t i = 0; i < m * k; ++i)
    x[i] = (float)((int64_t)(next_u64() % 2001) - 1000) / 37.0f;
  int8_t* q = malloc((size_t)(m * k));
  float* sx = malloc(sizeof(float) * (size_t)m);
  oracle_quantize_act(x, m, k, q, sx);
  int32_t* acc = malloc(sizeof(int32_t) * (size_t)(m * n));
  int32_t* acc4 = malloc(sizeof(int32_t) * (size_t)(m * n));
  oracle_gemm_i32(q, t, m, n, k, acc, 1);
  oracle_gemm_i32(q, t, m, n, k, acc4, 4);
  CHECK(memcmp(acc, acc4, sizeof(int32_t) * (size_t)(m * n)) == 0);
  CHECK(oracle_dot_i32(q + (m - 1) * k, t + (n - 1) * k, k) == acc[m * n - 1]);
  double* y = malloc(sizeof(double) * (size_t)(m * n));
  float* sw = malloc(sizeof(float) * (size_t)n);
  for (int64_t j = 0; j < n; ++j) sw[j] = 0.02f;
  oracle_epilogue(acc, sx, 0.02f, m, n, y);
  double* y2 = malloc(sizeof(double) * (size_t)(m * n));
  oracle_epilogue_rows(acc, sx, sw, m, n, y2);
  CHECK(memcmp(y, y2, sizeof(double) * (size_t)(m * n)) == 0);

  float* w = malloc(sizeof(float) * (size_t)(n * k));
  for (int64_t i = 0; i < n * k; ++i) w[i] = (float)((int64_t)(next_u64() % 201) - 100) / 64.0f;
  double* alpha = malloc(sizeof(double) * (size_t)n);
  const double a = oracle_ternarize(w, n, k, t2);
  oracle_ternarize_rows(w, n, k, t, alpha);
  CHECK(memcmp(t, t2, (size_t)(n * k)) == 0);
  CHECK(a >= 0.0 && !isnan(a));
  CHECK(oracle_pack(t, n, k, p) == 0); /* the ternarized matrix is 3:4 */
  free(t); free(t2); free(p); free(p2); free(x); free(q); free(sx); free(acc); free(acc4);
  free(y); free(y2); free(sw); free(w); free(alpha);
  return 0;
}

int main(void) {
  int8_t w[4];
  for (int c = 0; c < 32; ++c) {
    oracle_decode_code(c, w);
    if (oracle_encode_block(w) != c) return 1;
  }
  const int64_t shapes[][3] = {{1, 1, 4}, {3, 65, 132}, {2, 130, 516}, {5, 64, 2048},
                               {1, 7, 12}, {4, 200, 1028}};
  for (size_t i = 0; i < sizeof(shapes) / sizeof(shapes[0]); ++i)
    if (one_shape(shapes[i][0], shapes[i][1], shapes[i][2])) return 1;
  /* a block with two zeros is not 3:4: the packer rejects it */
  int8_t bad[8] = {0, 0, 1, 1, 0, 1, 1, 1};
  uint8_t* out = malloc((size_t)oracle_packed_bytes(1, 8)); /* one whole 1280-byte unit */
  if (oracle_pack(bad, 1, 8, out) != -1) return 1;        /* block 0 */
  free(out);
  puts("oracle sanitizer driver: ok");
  return 0;
}
