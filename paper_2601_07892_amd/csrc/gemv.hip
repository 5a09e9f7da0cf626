// Decode-path product for M <= 4 tokens (online phase of Appendix A, Eq. 2).
//
// Work mapping.  A workgroup is kGemvWaves waves; lane i of a wave owns row
// 64*r + i of one 64-row tile r, so the activations of a container (128
// weights) are the same for the whole wave and are read with scalar loads
// into SGPRs.
// Each tile's containers are split among S = gemv_split(C) waves (a power of
// two, so that a wave streams a few containers); a workgroup covers
// kGemvWaves/S tiles and its waves combine their int32 partial sums through
// LDS.
//
// Streaming.  A container is two contiguous wave-wide loads: the 64 rows'
// 16-byte heads (1 KB) and 4-byte tails (256 B).  Each wave keeps a ring of
// kRing containers in registers, refilling each slot as soon as it has been
// decoded.
//
// Decode.  Per code: a funnel shift and mask (or one SDWA mask) give code*4,
// one LDS read of the 32-entry table gives the int8x4 weights, one v_dot4 per
// token accumulates x . w in int32.  The table holds one dword per code, so
// any 64 lookups are free of bank conflicts.  The fused quantize + product
// kernels (one token) accumulate on the matrix cores instead of with v_dot4
// (dot_container_mfma).
//
// Lane-interleaved units (sherry_pack_il): the same stream, with each lane's
// 4-code chunks arranged as B operands of v_mfma_i32_16x16x64_i8 over 16 rows
// and 64 weights (dot_il), so that one activation operand per half unit
// serves all four row groups; the fused one-token step and the grouped
// products of up to four tokens have variants on them.
#include <type_traits>
#include <utility>

#include "sherry_internal.h"

namespace sherry {
namespace {

constexpr int kGemvThreads = 64 * kGemvWaves;
constexpr int kRing = 3;  // containers per wave held in the register ring
// The lane-interleaved decode keeps one container in flight beside the one
// it decodes: measured 1-2% faster than three on the LLaMA-3.2-1B step (less
// of the stream queued ahead of the workgroups that start late).
constexpr int kIlRing = 2;

typedef int v4i __attribute__((ext_vector_type(4)));

template <int j0, int... js>
__device__ __forceinline__ void group_offsets(const uint32_t (&d)[5], uint32_t* a4,
                                              std::integer_sequence<int, js...>) {
  ((a4[js] = code_x4<j0 + js>(d)), ...);
}

// Codes decoded per batch of table reads: all 32 of a container for one
// token (one wait for 32 table reads in flight); 8 when several tokens'
// activation words must sit in SGPRs at once.
template <int M>
constexpr int group_size() { return M == 1 ? 32 : 8; }

// Decodes codes [g, g + G) of a container in d[0..4] and accumulates the dot
// products with the activation words at xw (M tokens, row stride kw words,
// wave-uniform: scalar loads into SGPRs).  Words at or beyond words_left read
// as zero (last, partial container).
template <int M, bool kTail, int g = 0>
__device__ __forceinline__ void dot_container(const uint32_t (&d)[5],
                                              const SHERRY_CONST int32_t* xw, int kw,
                                              int words_left, const uint32_t* lut,
                                              int32_t (&acc)[M]) {
  constexpr int G = group_size<M>();
  if constexpr (g < 32) {
    // keep each group's loads, table reads and dot products together: the
    // scheduler would otherwise hoist every group's loads and run out of
    // scalar registers
    __builtin_amdgcn_sched_barrier(0);
    int32_t xv[M][G];
#pragma unroll
    for (int m = 0; m < M; ++m)
#pragma unroll
      for (int j = 0; j < G; ++j) {
        if constexpr (kTail) {
          // branch-free: read an in-bounds word, then zero it past K
          const int idx = (g + j < words_left) ? g + j : words_left - 1;
          const int32_t v = xw[m * kw + idx];
          xv[m][j] = (g + j < words_left) ? v : 0;
        } else {
          xv[m][j] = xw[m * kw + g + j];
        }
      }
    uint32_t a4[G];
    group_offsets<g>(d, a4, std::make_integer_sequence<int, G>{});
    uint32_t wv[G];
#pragma unroll
    for (int j = 0; j < G; ++j)
      wv[j] = *reinterpret_cast<const uint32_t*>(reinterpret_cast<const char*>(lut) + a4[j]);
#pragma unroll
    for (int j = 0; j < G; ++j)
#pragma unroll
      for (int m = 0; m < M; ++m)
        acc[m] = __builtin_amdgcn_sdot4(xv[m][j], static_cast<int32_t>(wv[j]), acc[m], false);
    dot_container<M, kTail, g + G>(d, xw, kw, words_left, lut, acc);
  }
}

// Decodes codes [g, g + 16) of a container and accumulates them against the
// activation words at xv (LDS, 16-byte aligned; zero past K).
template <int g>
__device__ __forceinline__ void dot_container_lds(const uint32_t (&d)[5], const u32x4* xv,
                                                  const uint32_t* lut, int32_t (&acc)[1]) {
  if constexpr (g < 32) {
    __builtin_amdgcn_sched_barrier(0);
    u32x4 xw[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) xw[i] = xv[g / 4 + i];
    uint32_t a4[16];
    group_offsets<g>(d, a4, std::make_integer_sequence<int, 16>{});
    uint32_t wv[16];
#pragma unroll
    for (int j = 0; j < 16; ++j)
      wv[j] = *reinterpret_cast<const uint32_t*>(reinterpret_cast<const char*>(lut) + a4[j]);
#pragma unroll
    for (int j = 0; j < 16; ++j)
      acc[0] = __builtin_amdgcn_sdot4(static_cast<int32_t>(xw[j >> 2][j & 3]),
                                      static_cast<int32_t>(wv[j]), acc[0], false);
    dot_container_lds<g + 16>(d, xv, lut, acc);
  }
}

// One token on the matrix cores: decodes codes [g, g + 16) of a container and
// accumulates them with v_mfma_i32_16x16x64_i8.  Lane 16b + t holds row
// 16b + t of the tile, so the looked-up words of a 4-code chunk (16 weights)
// are the B operand as they stand: column t, k block b.  The A operand is the
// chunk's 16 activations in lane 16b + b (A row b, k block b) and zeros in
// every other lane, so D[i][t] sums row 16i + t of the tile and nothing else
// (rows i >= 4 of D stay zero).  Only the lanes with own set read the
// activations at xv into xw; the other lanes' xw hold zeros throughout.  Two
// accumulators take alternate chunks; with kChain one accumulator takes all
// of them, starting from zero (a container's sum on its own).
template <int g, bool kChain = false>
__device__ __forceinline__ void dot_container_mfma(const uint32_t (&d)[5], const u32x4* xv,
                                                   bool own, u32x4 (&xw)[4], const uint32_t* lut,
                                                   v4i (&acc)[2]) {
  if constexpr (g < 32) {
    __builtin_amdgcn_sched_barrier(0);
    if (own) {
#pragma unroll
      for (int i = 0; i < 4; ++i) xw[i] = xv[g / 4 + i];
    }
    uint32_t a4[16];
    group_offsets<g>(d, a4, std::make_integer_sequence<int, 16>{});
    uint32_t wv[16];
#pragma unroll
    for (int j = 0; j < 16; ++j)
      wv[j] = *reinterpret_cast<const uint32_t*>(reinterpret_cast<const char*>(lut) + a4[j]);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const v4i a = {static_cast<int>(xw[q].x), static_cast<int>(xw[q].y),
                     static_cast<int>(xw[q].z), static_cast<int>(xw[q].w)};
      const v4i b = {static_cast<int>(wv[4 * q]), static_cast<int>(wv[4 * q + 1]),
                     static_cast<int>(wv[4 * q + 2]), static_cast<int>(wv[4 * q + 3])};
      if constexpr (kChain) {
        const v4i cin = (g == 0 && q == 0) ? v4i{0, 0, 0, 0} : acc[0];
        acc[0] = __builtin_amdgcn_mfma_i32_16x16x64_i8(a, b, cin, 0, 0, 0);
      } else {
        acc[q & 1] = __builtin_amdgcn_mfma_i32_16x16x64_i8(a, b, acc[q & 1], 0, 0, 0);
      }
    }
    dot_container_mfma<g + 16, kChain>(d, xv, own, xw, lut, acc);
  }
}

// Activation source: the activation words of container c, read with scalar
// loads (wave-uniform) into SGPRs; dot masks the words past K of a partial
// last container.
template <int M>
struct XFromSgpr {
  const SHERRY_CONST int32_t* xw0;  // [M][k/4] words in global memory
  int k;
  __device__ __forceinline__ void dot_full(const uint32_t (&d)[5], int c, const uint32_t* lut,
                                           int32_t (&acc)[M]) const {
    dot_container<M, false>(d, xw0 + c * (kTileK / 4), k >> 2, 32, lut, acc);
  }
  __device__ __forceinline__ void dot(const uint32_t (&d)[5], int c, const uint32_t* lut,
                                      int32_t (&acc)[M]) const {
    const int kb = c * kTileK;
    if (kb + kTileK <= k) dot_full(d, c, lut, acc);
    else dot_container<M, true>(d, xw0 + (kb >> 2), k >> 2, (k - kb) >> 2, lut, acc);
  }
};

// Activation source of the fused quantize + product kernel: the int8 words
// of the whole (zero-padded) activation row in LDS, read with wave-uniform
// 16-byte LDS loads (broadcast) in groups of 16 codes.
struct XFromLds {
  const int8_t* xq;  // LDS, ceil(k/128)*128 bytes
  __device__ __forceinline__ void dot(const uint32_t (&d)[5], int c, const uint32_t* lut,
                                      int32_t (&acc)[1]) const {
    dot_container_lds<0>(d, reinterpret_cast<const u32x4*>(xq + c * kTileK), lut, acc);
  }
};

// The same activations as the A operand of dot_container_mfma: lanes 16b + b
// read container c's words from xq (exec-masked LDS reads of 4 lanes); the
// other lanes' registers keep the zeros they start with.
struct XFromLdsMfma {
  const int8_t* xq;  // LDS, ceil(k/128)*128 bytes
  mutable u32x4 xw[4] = {};
  __device__ __forceinline__ void dot(const uint32_t (&d)[5], int c, const uint32_t* lut,
                                      v4i (&acc)[2]) const {
    const int lane = threadIdx.x & 63;
    dot_container_mfma<0>(d, reinterpret_cast<const u32x4*>(xq + c * kTileK),
                          (lane & 15) == (lane >> 4), xw, lut, acc);
  }
};

// Up to four tokens on the matrix cores, with the same B operand (lane
// 16b + t holds row 16b + t of the tile): A row 4b + m carries token m's
// chunk in k block b, so D[4b + m][t] = x_m . w(row 16b + t), and lane
// 16b + t ends with its own row's token sums in its accumulator elements
// 0..M-1.  The A operand of lane 20b + m (m < M) is read from token m's row
// of xq; every other lane's stays zero.  The matrix-core work per container
// is the same for one to four tokens.
struct XFromLdsMfmaTok {
  const int8_t* xq;  // LDS, M rows of kp bytes (zero past k)
  int kp, m_count;
  mutable u32x4 xw[4] = {};
  __device__ __forceinline__ void dot(const uint32_t (&d)[5], int c, const uint32_t* lut,
                                      v4i (&acc)[2]) const {
    const int lane = threadIdx.x & 63;
    const int m = (lane & 15) - 4 * (lane >> 4);
    const bool own = m >= 0 && m < m_count;
    dot_container_mfma<0>(d, reinterpret_cast<const u32x4*>(xq + (own ? m : 0) * kp + c * kTileK),
                          own, xw, lut, acc);
  }
  // container c's sums alone, in acc[0]
  __device__ __forceinline__ void dot_one(const uint32_t (&d)[5], int c, const uint32_t* lut,
                                          v4i (&acc)[2]) const {
    const int lane = threadIdx.x & 63;
    const int m = (lane & 15) - 4 * (lane >> 4);
    const bool own = m >= 0 && m < m_count;
    dot_container_mfma<0, true>(
        d, reinterpret_cast<const u32x4*>(xq + (own ? m : 0) * kp + c * kTileK), own, xw, lut,
        acc);
  }
};

// Lane-interleaved units (sherry_pack_il): lane 16b + t holds, as its codes
// 4(2g + p) .. 4(2g + p) + 3, row 16g + t's 16 weights of chunk 4p + b
// (g, b = 0..3; p = 0, 1).  So for chunk slot (g, p) the looked-up words are
// the B operand of one v_mfma_i32_16x16x64_i8 over 16 rows (16g + t, column
// t) and 64 weights (chunks 4p .. 4p + 3, k block b), and the A operand,
// token m's activations of those chunks in lanes 16b + m, serves all four
// row groups: two 16-byte activation reads per container instead of eight.
// D[m][t] = x_m . w(16g + t) lands in lane 16(m/4) + t, element m % 4 of
// accumulator g.
template <int G2>
__device__ __forceinline__ void dot_il(const uint32_t (&d)[5], const u32x4 (&xa)[2],
                                       const uint32_t* lut, v4i (&acc)[4]) {
  __builtin_amdgcn_sched_barrier(0);
  uint32_t a4[16];
  group_offsets<16 * G2>(d, a4, std::make_integer_sequence<int, 16>{});
  uint32_t wv[16];
#pragma unroll
  for (int j = 0; j < 16; ++j)
    wv[j] = *reinterpret_cast<const uint32_t*>(reinterpret_cast<const char*>(lut) + a4[j]);
  // slots (g, p) = (2 G2 + (s >> 1), s & 1), issued alternating accumulators
  constexpr int order[4] = {0, 2, 1, 3};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int s = order[i];
    const int g = 2 * G2 + (s >> 1), p = s & 1;
    const v4i a = {static_cast<int>(xa[p].x), static_cast<int>(xa[p].y),
                   static_cast<int>(xa[p].z), static_cast<int>(xa[p].w)};
    const v4i b = {static_cast<int>(wv[4 * s]), static_cast<int>(wv[4 * s + 1]),
                   static_cast<int>(wv[4 * s + 2]), static_cast<int>(wv[4 * s + 3])};
    acc[g] = __builtin_amdgcn_mfma_i32_16x16x64_i8(a, b, acc[g], 0, 0, 0);
  }
}

// Activation source of the lane-interleaved units: up to 16 token rows in
// LDS (kp bytes each, zero past k); lanes 16b + m with m < m_count read token
// m's chunks b and 4 + b of the container, every other lane keeps zeros.
struct XFromLdsMfmaIL {
  const int8_t* xq;
  int kp, m_count;
  mutable u32x4 xa[2] = {};
  __device__ __forceinline__ void dot(const uint32_t (&d)[5], int c, const uint32_t* lut,
                                      v4i (&acc)[4]) const {
    const int lane = threadIdx.x & 63;
    const int m = lane & 15, b = lane >> 4;
    if (m < m_count) {
      const u32x4* xv = reinterpret_cast<const u32x4*>(xq + m * kp + c * kTileK);
      xa[0] = xv[b];
      xa[1] = xv[4 + b];
    }
    dot_il<0>(d, xa, lut, acc);
    dot_il<1>(d, xa, lut, acc);
  }
};

template <class X>
constexpr bool kMfmaSource = false;
template <>
constexpr bool kMfmaSource<XFromLdsMfma> = true;
template <>
constexpr bool kMfmaSource<XFromLdsMfmaTok> = true;
template <>
constexpr bool kMfmaSource<XFromLdsMfmaIL> = true;

// Streams containers [c0, c1) of one tile through a ring of kRing register
// slots: slot u is decoded and immediately refilled with the container kRing
// ahead, so kRing - 1 containers are always in flight.  The run spans exactly
// [c0, c1) (container indices are relative to c0): refills past the end are
// issued unconditionally and read zeros without touching memory, which keeps
// the outstanding loads identical on every path so the compiler waits on
// exact counts; only the decode is skipped past the end.
// ring_fill issues the first R containers; ring_run decodes them all.  R is
// kRing except on lane-interleaved units, whose decode takes a ring of two
// (kIlRing).
template <int R>
__device__ __forceinline__ void ring_fill(uint32_t (&ring)[R][5], const UnitRun& run) {
  const int lane = threadIdx.x & 63;
  // issue the slots strictly in order (head and tail of slot 0 first), so
  // that slot u's loads are always the oldest outstanding ones when it is
  // decoded
#pragma unroll
  for (int u = 0; u < R; ++u) {
    load_unit(ring[u], run, u, lane);
    __builtin_amdgcn_sched_barrier(0);
  }
}

template <int R, class X, class Acc>
__device__ __forceinline__ void ring_run(uint32_t (&ring)[R][5], const UnitRun& run,
                                         int c0, int c1, const X& xsrc, const uint32_t* lut,
                                         Acc& acc) {
  const int lane = threadIdx.x & 63;
  const int n = c1 - c0;
  for (int i = 0; i < n; i += R) {
#pragma unroll
    for (int u = 0; u < R; ++u) {
      if (i + u < n) xsrc.dot(ring[u], c0 + i + u, lut, acc);
      __builtin_amdgcn_sched_barrier(0);
      load_unit(ring[u], run, i + u + R, lane);
      __builtin_amdgcn_sched_barrier(0);
    }
  }
}

// Per-group scales (one per output row and 128 weights along K, i.e. per
// container): the same ring, plus one 4-byte scale per lane and container
// loaded with it through a resource over the tile's rows of the [n][G] scale
// matrix.  Each container's int32 sum is scaled into an fp32 accumulator
// (ascending container order) and also added to the int32 total.
__device__ __forceinline__ float load_group_scale(__amdgpu_buffer_rsrc_t gr, int G, int c,
                                                  int lane) {
  return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(gr, 4 * (lane * G + c), 0, 0));
}

template <int M, class X>
__device__ __forceinline__ void ring_run_groups(uint32_t (&ring)[kRing][5],
                                                const UnitRun& run,
                                                __amdgpu_buffer_rsrc_t gr, int G, int c0, int c1,
                                                const X& xsrc, const uint32_t* lut,
                                                int32_t (&acc)[M], float (&accf)[M]) {
  const int lane = threadIdx.x & 63;
  const int n = c1 - c0;
  float gring[kRing];
#pragma unroll
  for (int u = 0; u < kRing; ++u) gring[u] = load_group_scale(gr, G, c0 + u, lane);
  for (int i = 0; i < n; i += kRing) {
#pragma unroll
    for (int u = 0; u < kRing; ++u) {
      if (i + u < n) {
        int32_t a[M];
#pragma unroll
        for (int m = 0; m < M; ++m) a[m] = 0;
        xsrc.dot(ring[u], c0 + i + u, lut, a);
#pragma unroll
        for (int m = 0; m < M; ++m) {
          accf[m] = __builtin_fmaf(static_cast<float>(a[m]), gring[u], accf[m]);
          acc[m] += a[m];
        }
      }
      __builtin_amdgcn_sched_barrier(0);
      load_unit(ring[u], run, i + u + kRing, lane);
      gring[u] = load_group_scale(gr, G, c0 + i + u + kRing, lane);
      __builtin_amdgcn_sched_barrier(0);
    }
  }
}

// Per-group scales on the 4-token matrix-core source: each container's MFMAs
// run as one chain from zero (slot u of the ring accumulates in pend[u]),
// and the lane's own row's M token sums (elements 0..M-1) are scaled by the
// row's group scale into fp32 accumulators (ascending container order) and
// added to the int32 totals, as in ring_run_groups.  A container is scaled
// one step after its MFMAs were issued, once the next container's are in
// flight, so the chain's latency is not waited for; the walk runs one step
// past the last container for that (its loads read zeros).
template <int M, class X>
__device__ __forceinline__ void ring_run_groups_mfma(uint32_t (&ring)[kRing][5],
                                                     const UnitRun& run,
                                                     __amdgpu_buffer_rsrc_t gr, int G, int c0,
                                                     int c1, const X& xsrc, const uint32_t* lut,
                                                     int32_t (&acc)[M], float (&accf)[M]) {
  const int lane = threadIdx.x & 63;
  const int n = c1 - c0;
  float gring[kRing], gpend[kRing] = {};
  v4i pend[kRing][2] = {};
#pragma unroll
  for (int u = 0; u < kRing; ++u) gring[u] = load_group_scale(gr, G, c0 + u, lane);
  for (int i = 0; i <= n; i += kRing) {
#pragma unroll
    for (int u = 0; u < kRing; ++u) {
      const int j = i + u;
      if (j < n) {
        xsrc.dot_one(ring[u], c0 + j, lut, pend[u]);
        gpend[u] = gring[u];
      }
      // container j - 1, in the previous slot
      const int pu = (u + kRing - 1) % kRing;  // a constant once unrolled
      if (j >= 1 && j <= n) {
#pragma unroll
        for (int m = 0; m < M; ++m) {
          const int32_t a = pend[pu][0][m];
          accf[m] = __builtin_fmaf(static_cast<float>(a), gpend[pu], accf[m]);
          acc[m] += a;
        }
      }
      __builtin_amdgcn_sched_barrier(0);
      load_unit(ring[u], run, j + kRing, lane);
      gring[u] = load_group_scale(gr, G, c0 + j + kRing, lane);
      __builtin_amdgcn_sched_barrier(0);
    }
  }
}

// The same with 16-byte scale loads: a ring of four containers, and lane l
// reads the scales of its row for four containers at once (one load per
// round of four, issued two rounds ahead), which touches a quarter of the
// cache lines of one 4-byte load per container.  Needs every row's scales
// 16-byte aligned (G % 4 == 0, gs 16-byte aligned) and c0 % 4 == 0.
constexpr int kGRing = 4;

template <int M, class X>
__device__ __forceinline__ void ring_run_groups_mfma4(const UnitRun& run,
                                                      __amdgpu_buffer_rsrc_t gr, int G, int c0,
                                                      int c1, const X& xsrc, const uint32_t* lut,
                                                      int32_t (&acc)[M], float (&accf)[M]) {
  const int lane = threadIdx.x & 63;
  const int n = c1 - c0;
  uint32_t ring[kGRing][5];
#pragma unroll
  for (int u = 0; u < kGRing; ++u) {
    load_unit(ring[u], run, u, lane);
    __builtin_amdgcn_sched_barrier(0);
  }
  // scales of rounds 0 and 1 (containers c0 .. c0 + 7 of the lane's row)
  u32x4 gq0 = __builtin_amdgcn_raw_buffer_load_b128(gr, 4 * (lane * G + c0), 0, 0);
  u32x4 gq1 = __builtin_amdgcn_raw_buffer_load_b128(gr, 4 * (lane * G + c0 + kGRing), 0, 0);
  // sums and scale of the current and the previous container
  float gpend[2] = {0.0f, 0.0f};
  v4i pend[2][2] = {};
  for (int i = 0; i <= n; i += kGRing) {
    const u32x4 gcur = gq0;
    gq0 = gq1;
    gq1 = __builtin_amdgcn_raw_buffer_load_b128(gr, 4 * (lane * G + c0 + i + 2 * kGRing), 0, 0);
#pragma unroll
    for (int u = 0; u < kGRing; ++u) {
      const int j = i + u;
      if (j < n) {
        xsrc.dot_one(ring[u], c0 + j, lut, pend[u & 1]);
        const uint32_t gbits = gcur[u];  // (a bit cast of the element itself
                                         // reads element 0 with this compiler)
        gpend[u & 1] = __uint_as_float(gbits);
      }
      // container j - 1, in the previous slot
      const int pu = (u + 1) & 1;  // a constant once unrolled (kGRing is even)
      if (j >= 1 && j <= n) {
#pragma unroll
        for (int m = 0; m < M; ++m) {
          const int32_t a = pend[pu][0][m];
          accf[m] = __builtin_fmaf(static_cast<float>(a), gpend[pu], accf[m]);
          acc[m] += a;
        }
      }
      __builtin_amdgcn_sched_barrier(0);
      load_unit(ring[u], run, j + kGRing, lane);
      __builtin_amdgcn_sched_barrier(0);
    }
  }
}

// One workgroup of a product: block g of a problem whose tiles are split
// over S waves each.  prelude.issue() then prelude.finish(sx) run before the
// weight stream; finish yields the tokens' activation scales sx[m].  lut and red are
// LDS; the caller has filled lut.
//
// With kGrp the weights carry per-group scales gs ([n][ceil(k/128)] fp32):
// y = sx * sum over containers of float(acc_c) * gs[row][c], summed in fp32
// in container order per wave and then over the S waves in order; redf is
// LDS for the fp32 partial sums.
template <int M, bool kGrp = false, class X, class Prelude>
__device__ __forceinline__ void gemv_block(const uint8_t* w_, const X& xsrc, Prelude prelude,
                                           WScale ws, float* y, int32_t* acc_out, int64_t n,
                                           int k, int g, int S, const uint32_t* lut,
                                           int32_t* red, const float* gs = nullptr,
                                           float* redf = nullptr) {
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int C = (k + kTileK - 1) / kTileK;
  const int R = static_cast<int>((n + kTileRows - 1) / kTileRows);
  const int tpb = kGemvWaves / S;  // tiles per block
  const int lt = wave / S;         // tile of this wave inside the block
  const int part = wave - lt * S;  // part of the tile's containers
  const int r = g * tpb + lt;
  int32_t acc[M];
#pragma unroll
  for (int m = 0; m < M; ++m) acc[m] = 0;
  // a wave past the last tile streams an empty range (its loads read zeros)
  const int c0 = (r < R) ? (part * C) / S : 0, c1 = (r < R) ? ((part + 1) * C) / S : 0;
  const UnitRun range{w_ + (int64_t(r < R ? r : 0) * C + c0) * kUnitBytes, c1 - c0};
  // the prelude (e.g. quantizing the activations) runs to completion before
  // the first weight loads: its few loads then do not queue behind the
  // weight stream of every wave on the GPU; every thread of the block runs it
  prelude.issue();
  float sx[M];
  prelude.finish(sx);
  // the per-channel scales of this thread's outputs (output t = threadIdx.x
  // + j * kGemvThreads: row 64 (g tpb + (t / 64) / M) + t % 64) are loaded
  // now: their latency hides behind the stream instead of ending the
  // workgroup, and no load sits between the epilogue's stores (one counter
  // tracks a wave's loads and stores, so it would wait for every store
  // before it)
  constexpr int kOut = (kGemvWaves * M * 64 + kGemvThreads - 1) / kGemvThreads;
  float swo[kOut];
#pragma unroll
  for (int j = 0; j < kOut; ++j) {
    const int t = static_cast<int>(threadIdx.x) + j * kGemvThreads;
    const int r0 = g * tpb + (t >> 6) / M;
    const int64_t row0 = int64_t(r0) * kTileRows + (t & 63);
    swo[j] = (ws.rows && t < tpb * M * 64 && r0 < R && row0 < n) ? as_global(ws.rows)[row0]
                                                                  : ws.tensor;
  }
  __builtin_amdgcn_sched_barrier(0);
  float accf[M];
  if constexpr (kGrp) {
    // scale rows of this wave's tile (rows past n read zero)
    const int rows = (r < R) ? static_cast<int>(n - int64_t(r) * kTileRows) : 0;
    const __amdgpu_buffer_rsrc_t gr = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<float*>(gs) + int64_t(r < R ? r : 0) * kTileRows * C, 0,
        (rows < kTileRows ? rows : kTileRows) * C * 4, kBufferWord3);
#pragma unroll
    for (int m = 0; m < M; ++m) accf[m] = 0.0f;
    if constexpr (kMfmaSource<X>) {
      static_assert(std::is_same_v<X, XFromLdsMfmaTok>,
                    "per-group scales on the matrix cores: the token source only");
      if (C % 4 == 0 && (reinterpret_cast<uintptr_t>(gs) & 15) == 0) {
        // 16-byte scale loads: the parts of the tile start at multiples of
        // four containers
        auto bound = [&](int p) { return p >= S ? C : ((p * C) / S) & ~3; };
        const int b0 = (r < R) ? bound(part) : 0, b1 = (r < R) ? bound(part + 1) : 0;
        const UnitRun run4{w_ + (int64_t(r < R ? r : 0) * C + b0) * kUnitBytes, b1 - b0};
        ring_run_groups_mfma4<M>(run4, gr, C, b0, b1, xsrc, lut, acc, accf);
      } else {
        uint32_t ring[kRing][5];
        ring_fill(ring, range);
        ring_run_groups_mfma<M>(ring, range, gr, C, c0, c1, xsrc, lut, acc, accf);
      }
      // the LDS of the activations is reused: every wave has finished reading it
      __syncthreads();
#pragma unroll
      for (int m = 0; m < M; ++m) red[(wave * M + m) * 64 + lane] = acc[m];
    } else {
      uint32_t ring[kRing][5];
      ring_fill(ring, range);
      ring_run_groups<M>(ring, range, gr, C, c0, c1, xsrc, lut, acc, accf);
    }
  } else if constexpr (std::is_same_v<X, XFromLdsMfmaIL>) {
    static_assert(M <= 4, "the lane-interleaved source serves up to four tokens here");
    uint32_t ring[kIlRing][5];
    ring_fill(ring, range);
    v4i macc[4] = {};
    ring_run(ring, range, c0, c1, xsrc, lut, macc);
    // lane l < 16 holds token m of row 16g + l of the tile in element m of
    // accumulator g; red may be the LDS of the staged rows, reused once every
    // wave has finished reading it
    __syncthreads();
    if (lane < 16) {
#pragma unroll
      for (int g = 0; g < 4; ++g)
#pragma unroll
        for (int m = 0; m < M; ++m) red[(wave * M + m) * 64 + 16 * g + lane] = macc[g][m];
    }
  } else if constexpr (kMfmaSource<X>) {
    static_assert(M <= 4 && !kGrp, "the matrix-core sources serve up to four tokens");
    uint32_t ring[kRing][5];
    ring_fill(ring, range);
    v4i macc[2] = {{0, 0, 0, 0}, {0, 0, 0, 0}};
    ring_run(ring, range, c0, c1, xsrc, lut, macc);
    if constexpr (std::is_same_v<X, XFromLdsMfma>) {
      // lane l < 16 holds rows l, 16 + l, 32 + l, 48 + l of the tile
      if (lane < 16) {
#pragma unroll
        for (int e = 0; e < 4; ++e) red[wave * 64 + 16 * e + lane] = macc[0][e] + macc[1][e];
      }
    } else {
      // the LDS of the activations is reused: every wave has finished reading it
      __syncthreads();
#pragma unroll
      for (int m = 0; m < M; ++m) red[(wave * M + m) * 64 + lane] = macc[0][m] + macc[1][m];
    }
  } else {
    uint32_t ring[kRing][5];
    ring_fill(ring, range);
    ring_run(ring, range, c0, c1, xsrc, lut, acc);
  }

  if constexpr (!kMfmaSource<X>) {
#pragma unroll
    for (int m = 0; m < M; ++m) red[(wave * M + m) * 64 + lane] = acc[m];
  }
  if constexpr (kGrp) {
#pragma unroll
    for (int m = 0; m < M; ++m) redf[(wave * M + m) * 64 + lane] = accf[m];
  }
  __syncthreads();
  // the scales are waited for here, once, before the first store (a wait
  // inside the loop would also wait for the stores issued before it)
#pragma unroll
  for (int j = 0; j < kOut; ++j) asm volatile("" ::"v"(swo[j]));
  // thread t -> (tile lt2, token m, row i); the S waves of a tile are adjacent
#pragma unroll
  for (int j = 0; j < kOut; ++j) {
    const int t = static_cast<int>(threadIdx.x) + j * kGemvThreads;
    if (t >= tpb * M * 64) break;
    const int i = t & 63;
    const int m = (t >> 6) % M;
    const int lt2 = (t >> 6) / M;
    const int r2 = g * tpb + lt2;
    const int64_t row = int64_t(r2) * kTileRows + i;
    if (r2 >= R || row >= n) continue;
    int32_t a = 0;
    for (int p = 0; p < S; ++p) a += red[((lt2 * S + p) * M + m) * 64 + i];
    if constexpr (kGrp) {
      float f = 0.0f;
      for (int p = 0; p < S; ++p) f += redf[((lt2 * S + p) * M + m) * 64 + i];
      as_global_mut(y)[m * n + row] = f * sx[m];
    } else {
      const float s = sx[m] * swo[j];
      as_global_mut(y)[m * n + row] = static_cast<float>(a) * s;
    }
    if (acc_out) as_global_mut(acc_out)[m * n + row] = a;
  }
}

// Prelude of the int8 products: the activation scales are inputs.
template <int M>
struct ReadScales {
  const float* x_scale;
  __device__ __forceinline__ void issue() const {}
  __device__ __forceinline__ void finish(float (&sx)[M]) const {
#pragma unroll
    for (int m = 0; m < M; ++m) sx[m] = as_const(x_scale)[m];
  }
};

__device__ __forceinline__ void fill_lut(uint32_t* lut) {
  if (threadIdx.x < 32) lut[threadIdx.x] = decode_word(threadIdx.x);
}

// Block of a grouped launch that workgroup b runs.  Workgroups are dispatched
// to the 8 XCDs in turn (b -> XCD b % 8), each with its own L2; XCD x takes
// the x-th contiguous eighth of the blocks, so that the workgroups of one
// product meet in few L2s and its activation row is fetched there once.
__device__ __forceinline__ int32_t xcd_block(int32_t b, int32_t grid) {
  constexpr int32_t kXcds = 8;
  const int32_t q = grid / kXcds, r = grid % kXcds;
  const int32_t x = b % kXcds, slot = b / kXcds;
  return x < r ? x * (q + 1) + slot : r * (q + 1) + (x - r) * q + slot;
}

// Barrier for LDS traffic only: outstanding global loads (the weight ring)
// stay in flight across it.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Prelude of the matrix-core int8 products: copies the M activation rows
// (int8 [M][k], k % 4 == 0) into xq (LDS, rows of kp bytes, zero past k) and
// reads the tokens' scales.
// Largest M * kp (bytes of staged activations) of the matrix-core int8
// products: their LDS holds the rows and, after the stream, the partial sums.
constexpr int kTokMaxBytes = 32768;

template <int M>
struct StageRows {
  static constexpr int kPieces = kTokMaxBytes / 16 / kGemvThreads;  // per thread
  const int8_t* x;
  const float* x_scale;
  int k, kp;
  int8_t* xq;
  u32x4 v[kPieces];
  // Rows whose 16-byte pieces are aligned (k % 16 == 0, x 16-byte aligned)
  // are loaded as such, all of a thread's pieces in flight at once, and
  // stored by finish(); other rows are copied in 4-byte words by finish().
  __device__ __forceinline__ bool wide() const {
    return (k & 15) == 0 && (reinterpret_cast<uintptr_t>(x) & 15) == 0;
  }
  __device__ __forceinline__ void issue() {
    if (!wide()) return;
    const SHERRY_GLOBAL u32x4* x16 = as_global(reinterpret_cast<const u32x4*>(x));
    const int k16 = k >> 4, kp16 = kp >> 4;
#pragma unroll
    for (int e = 0; e < kPieces; ++e) {
      const int i = threadIdx.x + e * kGemvThreads;
      const int m = i / kp16, j = i - m * kp16;
      // every thread loads (an in-bounds piece when past the rows), so the
      // loads go out back to back
      const bool in = m < M && j < k16;
      const u32x4 t = x16[in ? m * k16 + j : 0];
      v[e] = in ? t : u32x4{0u, 0u, 0u, 0u};
    }
  }
  __device__ __forceinline__ void finish(float (&sx)[M]) {
    if (wide()) {
      u32x4* q16 = reinterpret_cast<u32x4*>(xq);
#pragma unroll
      for (int e = 0; e < kPieces; ++e) {
        const int i = threadIdx.x + e * kGemvThreads;
        if (i < M * (kp >> 4)) q16[i] = v[e];
      }
    } else {
      const SHERRY_GLOBAL uint32_t* x4 = as_global(reinterpret_cast<const uint32_t*>(x));
      uint32_t* q4 = reinterpret_cast<uint32_t*>(xq);
      const int k4 = k >> 2, kp4 = kp >> 2;
      for (int i = threadIdx.x; i < M * kp4; i += kGemvThreads) {
        const int m = i / kp4, j = i - m * kp4;
        q4[i] = j < k4 ? x4[m * k4 + j] : 0u;
      }
    }
#pragma unroll
    for (int m = 0; m < M; ++m) sx[m] = as_const(x_scale)[m];
    lds_barrier();
  }
};

// LDS of the 4-token kernels: the staged activation rows, which after the
// stream hold the int32 partial sums (first 8 KB) and, with per-group scales,
// the fp32 ones (next 8 KB).
static_assert(2 * kGemvWaves * 4 * 64 * 4 <= kTokMaxBytes, "partial sums fit the staging");
__device__ __forceinline__ float* tok_redf(int8_t* xq) {
  return reinterpret_cast<float*>(xq + kGemvWaves * 4 * 64 * 4);
}

template <int M, bool kGrp>
__global__ __launch_bounds__(kGemvThreads) void gemv_tok_kernel(
    const uint8_t* __restrict__ w, const int8_t* __restrict__ x,
    const float* __restrict__ x_scale, WScale ws, const float* __restrict__ gs,
    float* __restrict__ y, int32_t* __restrict__ acc, int64_t n, int64_t k, int split) {
  __shared__ uint32_t lut[32];
  __shared__ __attribute__((aligned(16))) int8_t xq[kTokMaxBytes];
  fill_lut(lut);
  const int kp = static_cast<int>((k + kTileK - 1) / kTileK) * kTileK;
  gemv_block<M, kGrp>(w, XFromLdsMfmaTok{xq, kp, M},
                      StageRows<M>{x, x_scale, static_cast<int>(k), kp, xq}, ws, y, acc, n,
                      static_cast<int>(k), blockIdx.x, split, lut,
                      reinterpret_cast<int32_t*>(xq), gs, tok_redf(xq));
}

template <int M, bool kGrp>
__device__ __forceinline__ void tok_batched_block(const sherry_gemm_desc& d, int g,
                                                  const uint32_t* lut, int8_t* xq) {
  const int k = static_cast<int>(d.k);
  const int kp = ((k + kTileK - 1) / kTileK) * kTileK;
  const int S = gemv_split((k + kTileK - 1) / kTileK);
  gemv_block<M, kGrp>(d.w, XFromLdsMfmaTok{xq, kp, M}, StageRows<M>{d.x, d.x_scale, k, kp, xq},
                      WScale{d.w_scales, d.w_scale}, d.y, d.acc, d.n, k, g, S, lut,
                      reinterpret_cast<int32_t*>(xq), d.w_group_scales, tok_redf(xq));
}

// The same on lane-interleaved weights (per-tensor and per-channel scales).
template <int M>
__device__ __forceinline__ void tok_il_batched_block(const sherry_gemm_desc& d, int g,
                                                     const uint32_t* lut, int8_t* xq) {
  const int k = static_cast<int>(d.k);
  const int kp = ((k + kTileK - 1) / kTileK) * kTileK;
  const int S = gemv_split((k + kTileK - 1) / kTileK);
  gemv_block<M>(d.w, XFromLdsMfmaIL{xq, kp, M}, StageRows<M>{d.x, d.x_scale, k, kp, xq},
                WScale{d.w_scales, d.w_scale}, d.y, d.acc, d.n, k, g, S, lut,
                reinterpret_cast<int32_t*>(xq));
}

// Grouped products of up to four tokens each on lane-interleaved weights
// (m * ceil(k/128) * 128 <= kTokMaxBytes, no per-group scales).
__global__ __launch_bounds__(kGemvThreads) void gemv_tok_il_batched_kernel(
    const sherry_gemm_desc* __restrict__ descs, int count) {
  __shared__ uint32_t lut[32];
  __shared__ __attribute__((aligned(16))) int8_t xq[kTokMaxBytes];
  fill_lut(lut);
  const int32_t blk = static_cast<int32_t>(blockIdx.x);
  const int lo = find_block_desc(descs, count, blk);
  if (lo < 0) return;
  const sherry_gemm_desc& d = descs[lo];
  const int g = blk - d.block_begin;
  switch (d.m) {
    case 1: tok_il_batched_block<1>(d, g, lut, xq); break;
    case 2: tok_il_batched_block<2>(d, g, lut, xq); break;
    case 3: tok_il_batched_block<3>(d, g, lut, xq); break;
    default: tok_il_batched_block<4>(d, g, lut, xq); break;
  }
}

// Grouped products of up to four tokens each (sherry_gemm_desc,
// m * ceil(k/128) * 128 <= kTokMaxBytes): per-tensor and per-channel scales,
// and with kGroups also per-group ones (a kernel of its own, so that the
// others keep the registers of the plain stream).
template <bool kGroups>
__global__ __launch_bounds__(kGemvThreads) void gemv_tok_batched_kernel(
    const sherry_gemm_desc* __restrict__ descs, int count) {
  __shared__ uint32_t lut[32];
  __shared__ __attribute__((aligned(16))) int8_t xq[kTokMaxBytes];
  fill_lut(lut);
  const int32_t blk = static_cast<int32_t>(blockIdx.x);
  const int lo = find_block_desc(descs, count, blk);
  if (lo < 0) return;
  const sherry_gemm_desc& d = descs[lo];
  const int g = blk - d.block_begin;
  if (kGroups && d.w_group_scales) {
    switch (d.m) {
      case 1: tok_batched_block<1, kGroups>(d, g, lut, xq); break;
      case 2: tok_batched_block<2, kGroups>(d, g, lut, xq); break;
      case 3: tok_batched_block<3, kGroups>(d, g, lut, xq); break;
      default: tok_batched_block<4, kGroups>(d, g, lut, xq); break;
    }
  } else {
    switch (d.m) {
      case 1: tok_batched_block<1, false>(d, g, lut, xq); break;
      case 2: tok_batched_block<2, false>(d, g, lut, xq); break;
      case 3: tok_batched_block<3, false>(d, g, lut, xq); break;
      default: tok_batched_block<4, false>(d, g, lut, xq); break;
    }
  }
}

template <int M>
__global__ __launch_bounds__(kGemvThreads) void gemv_kernel(
    const uint8_t* __restrict__ w, const int8_t* __restrict__ x,
    const float* __restrict__ x_scale, WScale ws, float* __restrict__ y,
    int32_t* __restrict__ acc, int64_t n, int64_t k, int split) {
  __shared__ uint32_t lut[32];
  __shared__ int32_t red[kGemvWaves * M * 64];
  fill_lut(lut);
  gemv_block<M>(w, XFromSgpr<M>{as_const(reinterpret_cast<const int32_t*>(x)), static_cast<int>(k)},
                ReadScales<M>{x_scale}, ws, y, acc, n, static_cast<int>(k), blockIdx.x, split,
                lut, red);
}

template <int M>
__global__ __launch_bounds__(kGemvThreads) void gemv_group_kernel(
    const uint8_t* __restrict__ w, const int8_t* __restrict__ x,
    const float* __restrict__ x_scale, const float* __restrict__ gs, float* __restrict__ y,
    int32_t* __restrict__ acc, int64_t n, int64_t k, int split) {
  __shared__ uint32_t lut[32];
  __shared__ int32_t red[kGemvWaves * M * 64];
  __shared__ float redf[kGemvWaves * M * 64];
  fill_lut(lut);
  gemv_block<M, true>(w,
                      XFromSgpr<M>{as_const(reinterpret_cast<const int32_t*>(x)),
                                   static_cast<int>(k)},
                      ReadScales<M>{x_scale}, WScale{nullptr, 0.0f}, y, acc, n,
                      static_cast<int>(k), blockIdx.x, split, lut, red, gs, redf);
}

__global__ __launch_bounds__(kGemvThreads) void gemv_batched_kernel(
    const sherry_gemv_desc* __restrict__ descs, int count) {
  __shared__ uint32_t lut[32];
  __shared__ int32_t red[kGemvWaves * 64];
  __shared__ float redf[kGemvWaves * 64];
  fill_lut(lut);
  const int32_t blk = xcd_block(static_cast<int32_t>(blockIdx.x), static_cast<int32_t>(gridDim.x));
  // last descriptor with block_begin <= blk: block_begin strictly increases,
  // so the descriptors that qualify form a prefix; each lane tests one
  // descriptor and the prefix length comes from a ballot (one load round
  // trip per 64 descriptors instead of a chain of dependent loads)
  const int lane = threadIdx.x & 63;
  int lo = 0;
  for (int base = 0; base < count; base += 64) {
    const int i = base + lane;
    const bool ok = i < count && as_global(descs)[i].block_begin <= blk;
    const uint64_t m = __ballot(ok);
    const int len = __popcll(m);
    lo = base + len - 1;
    if (len < 64) break;
  }
  lo = __builtin_amdgcn_readfirstlane(lo);
  const sherry_gemv_desc& d = descs[lo];
  const int k = static_cast<int>(d.k);
  const int S = gemv_split(static_cast<int>((k + kTileK - 1) / kTileK));
  const XFromSgpr<1> xs{as_const(reinterpret_cast<const int32_t*>(d.x)), k};
  if (d.w_group_scales) {
    gemv_block<1, true>(d.w, xs, ReadScales<1>{d.x_scale}, WScale{nullptr, 0.0f}, d.y, d.acc,
                        d.n, k, blk - d.block_begin, S, lut, red, d.w_group_scales, redf);
  } else {
    gemv_block<1>(d.w, xs, ReadScales<1>{d.x_scale}, WScale{d.w_scales, d.w_scale}, d.y, d.acc,
                  d.n, k, blk - d.block_begin, S, lut, red);
  }
}

// ---- fused per-token quantization + product (M = 1) ----

// Block-wide max of one value per thread (part: kGemvWaves floats of LDS).
__device__ __forceinline__ float block_max_f32(float v, float* part) {
  v = wave_max_f32(v);
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = v;
  lds_barrier();
  v = part[0];
#pragma unroll
  for (int i = 1; i < kGemvWaves; ++i) v = fmaxf(v, part[i]);
  return v;
}

// Prelude of the fused kernels: quantizes the fp32 row x[0..k) into xq
// (LDS, int8, zero-padded to kp bytes) exactly as the quantize kernel does;
// the scale (0 for an all-zero row) is written to *x_scale by one thread
// when write_scale.  Rows of up to NV*4*kGemvThreads values are loaded once
// into registers by issue(); NV = 0 reads longer rows twice in finish() (the
// second time from cache).
template <int NV>
struct QuantizeRow {
  const float* x;
  int k, kp;
  int8_t* xq;
  float* part;  // LDS, kGemvWaves floats
  float* x_scale;
  bool write_scale;
  float4 v[NV > 0 ? NV : 1];

  __device__ __forceinline__ void issue() {
    if constexpr (NV > 0) {
      const float4* x4 = reinterpret_cast<const float4*>(as_global(x));
#pragma unroll
      for (int e = 0; e < NV; ++e) {
        const int i = threadIdx.x + e * kGemvThreads;
        // every thread loads (a clamped index past the row), so that the
        // loads issue back to back instead of behind exec-masked branches
        const int k4 = k >> 2;
        const float4 t = x4[i < k4 ? i : k4 - 1];
        v[e] = (i < k4) ? t : make_float4(0.f, 0.f, 0.f, 0.f);
      }
    }
  }

  __device__ __forceinline__ void finish(float (&sx)[1]) {
    const float4* x4 = reinterpret_cast<const float4*>(as_global(x));
    const int k4 = k >> 2;
    uint32_t* q4 = reinterpret_cast<uint32_t*>(xq);
    float amax = 0.0f;
    if constexpr (NV > 0) {
#pragma unroll
      for (int e = 0; e < NV; ++e)
        amax = fmaxf(amax, fmaxf(fmaxf(fabsf(v[e].x), fabsf(v[e].y)),
                                 fmaxf(fabsf(v[e].z), fabsf(v[e].w))));
      amax = block_max_f32(amax, part);
      const float s = amax / 127.0f;
      const float rs = 1.0f / s;
#pragma unroll
      for (int e = 0; e < NV; ++e) {
        const int i = threadIdx.x + e * kGemvThreads;
        if (i < (kp >> 2)) q4[i] = (i < k4 && amax != 0.0f) ? quant4(v[e], s, rs) : 0u;
      }
    } else {
      for (int i = threadIdx.x; i < k4; i += kGemvThreads) {
        const float4 w = x4[i];
        amax = fmaxf(amax, fmaxf(fmaxf(fabsf(w.x), fabsf(w.y)), fmaxf(fabsf(w.z), fabsf(w.w))));
      }
      amax = block_max_f32(amax, part);
      const float s = amax / 127.0f;
      const float rs = 1.0f / s;
      for (int i = threadIdx.x; i < (kp >> 2); i += kGemvThreads)
        q4[i] = (i < k4 && amax != 0.0f) ? quant4(x4[i], s, rs) : 0u;
    }
    lds_barrier();
    sx[0] = amax == 0.0f ? 0.0f : amax / 127.0f;
    if (write_scale && threadIdx.x == 0 && x_scale) as_global_mut(x_scale)[0] = sx[0];
  }
};

// Fused product of one block: the row length picks the quantizer (rows up
// to 2048, 8192 and 16384 values from registers, longer ones in two passes).
template <bool kGrp = false, bool kIL = false>
__device__ __forceinline__ void fused_block(const uint8_t* w, const float* x, float* x_scale,
                                            bool write_scale, WScale ws, float* y,
                                            int32_t* acc, int64_t n, int k, int g, int S,
                                            const uint32_t* lut, int32_t* red, float* part,
                                            int8_t* xq, const float* gs = nullptr,
                                            float* redf = nullptr) {
  const int kp = ((k + kTileK - 1) / kTileK) * kTileK;
  // per-tensor and per-channel scales sum a tile row's containers in int32 on
  // the matrix cores; per-group scales need each container's sum per lane;
  // kIL: lane-interleaved units
  static_assert(!(kGrp && kIL), "per-group scales: tiled units only");
  const auto xsrc = [&] {
    if constexpr (kGrp) return XFromLds{xq};
    else if constexpr (kIL) return XFromLdsMfmaIL{xq, kp, 1};
    else return XFromLdsMfma{xq};
  }();
  if (kp <= 4 * kGemvThreads) {
    gemv_block<1, kGrp>(w, xsrc,
                        QuantizeRow<1>{x, k, kp, xq, part, x_scale, write_scale}, ws, y, acc,
                        n, k, g, S, lut, red, gs, redf);
  } else if (kp <= 16 * kGemvThreads) {
    gemv_block<1, kGrp>(w, xsrc,
                        QuantizeRow<4>{x, k, kp, xq, part, x_scale, write_scale}, ws, y, acc,
                        n, k, g, S, lut, red, gs, redf);
  } else if (kp <= 32 * kGemvThreads) {
    gemv_block<1, kGrp>(w, xsrc,
                        QuantizeRow<8>{x, k, kp, xq, part, x_scale, write_scale}, ws, y, acc,
                        n, k, g, S, lut, red, gs, redf);
  } else {
    gemv_block<1, kGrp>(w, xsrc,
                        QuantizeRow<0>{x, k, kp, xq, part, x_scale, write_scale}, ws, y, acc,
                        n, k, g, S, lut, red, gs, redf);
  }
}

__global__ __launch_bounds__(kGemvThreads) void gemv_f32_kernel(
    const uint8_t* __restrict__ w, const float* __restrict__ x, float* __restrict__ x_scale,
    WScale ws, float* __restrict__ y, int32_t* __restrict__ acc, int64_t n, int64_t k,
    int split) {
  __shared__ uint32_t lut[32];
  __shared__ int32_t red[kGemvWaves * 64];
  __shared__ float part[kGemvWaves];
  __shared__ __attribute__((aligned(16))) int8_t xq[kFusedMaxK];
  fill_lut(lut);
  fused_block(w, x, x_scale, blockIdx.x == 0, ws, y, acc, n, static_cast<int>(k), blockIdx.x,
              split, lut, red, part, xq);
}

__global__ __launch_bounds__(kGemvThreads) void gemv_f32_group_kernel(
    const uint8_t* __restrict__ w, const float* __restrict__ x, float* __restrict__ x_scale,
    const float* __restrict__ gs, float* __restrict__ y, int32_t* __restrict__ acc, int64_t n,
    int64_t k, int split) {
  __shared__ uint32_t lut[32];
  __shared__ int32_t red[kGemvWaves * 64];
  __shared__ float redf[kGemvWaves * 64];
  __shared__ float part[kGemvWaves];
  __shared__ __attribute__((aligned(16))) int8_t xq[kFusedMaxK];
  fill_lut(lut);
  fused_block<true>(w, x, x_scale, blockIdx.x == 0, WScale{nullptr, 0.0f}, y, acc, n,
                    static_cast<int>(k), blockIdx.x, split, lut, red, part, xq, gs, redf);
}

template <bool kIL>
__global__ __launch_bounds__(kGemvThreads) void gemv_f32_batched_kernel(
    const sherry_gemv_f32_desc* __restrict__ descs, int count) {
  __shared__ uint32_t lut[32];
  __shared__ int32_t red[kGemvWaves * 64];
  __shared__ float redf[kGemvWaves * 64];
  __shared__ float part[kGemvWaves];
  __shared__ __attribute__((aligned(16))) int8_t xq[kFusedMaxK];
  fill_lut(lut);
  const int32_t blk = xcd_block(static_cast<int32_t>(blockIdx.x), static_cast<int32_t>(gridDim.x));
  const int lane = threadIdx.x & 63;
  int lo = 0;
  for (int base = 0; base < count; base += 64) {
    const int i = base + lane;
    const bool ok = i < count && as_global(descs)[i].block_begin <= blk;
    const uint64_t m = __ballot(ok);
    const int len = __popcll(m);
    lo = base + len - 1;
    if (len < 64) break;
  }
  lo = __builtin_amdgcn_readfirstlane(lo);
  const sherry_gemv_f32_desc& d = descs[lo];
  const int k = static_cast<int>(d.k);
  const int C = (k + kTileK - 1) / kTileK;
  const int S = fused_split(C);
  if constexpr (kIL) {
    fused_block<false, true>(d.w, d.x, d.x_scale, blk == d.block_begin,
                             WScale{d.w_scales, d.w_scale}, d.y, d.acc, d.n, k,
                             blk - d.block_begin, S, lut, red, part, xq);
  } else if (d.w_group_scales) {
    fused_block<true>(d.w, d.x, d.x_scale, blk == d.block_begin, WScale{nullptr, 0.0f}, d.y,
                      d.acc, d.n, k, blk - d.block_begin, S, lut, red, part, xq,
                      d.w_group_scales, redf);
  } else {
    fused_block(d.w, d.x, d.x_scale, blk == d.block_begin, WScale{d.w_scales, d.w_scale}, d.y,
                d.acc, d.n, k, blk - d.block_begin, S, lut, red, part, xq);
  }
}

}  // namespace

int launch_gemv_valu(const uint8_t* w, const int8_t* x, const float* x_scale, WScale ws,
                     float* y, int32_t* acc, int64_t m, int64_t n, int64_t k, hipStream_t s) {
  const int64_t R = ceil_div(n, kTileRows);
  const int C = static_cast<int>(ceil_div(k, kTileK));
  // a lone launch has only this product to fill the GPU: split every tile
  // over all waves of a workgroup unless there are plenty of tiles
  const int S = (R * gemv_split(C) >= 4096) ? gemv_split(C) : kGemvWaves;
  const dim3 grid(static_cast<unsigned>(ceil_div(R * S, kGemvWaves)));
  const dim3 block(kGemvThreads);
  switch (m) {
    case 1: return launch(gemv_kernel<1>, grid, block, 0, s, w, x, x_scale, ws, y, acc, n, k, S);
    case 2: return launch(gemv_kernel<2>, grid, block, 0, s, w, x, x_scale, ws, y, acc, n, k, S);
    case 3: return launch(gemv_kernel<3>, grid, block, 0, s, w, x, x_scale, ws, y, acc, n, k, S);
    case 4: return launch(gemv_kernel<4>, grid, block, 0, s, w, x, x_scale, ws, y, acc, n, k, S);
    default: return SHERRY_E_SHAPE;
  }
}

bool gemv_tok_fits(int64_t m, int64_t k) {
  return m >= 1 && m <= 4 && m * ceil_div(k, kTileK) * kTileK <= kTokMaxBytes;
}

int launch_gemv_tok(const uint8_t* w, const int8_t* x, const float* x_scale, WScale ws,
                    const float* gs, float* y, int32_t* acc, int64_t m, int64_t n, int64_t k,
                    hipStream_t s) {
  if (!gemv_tok_fits(m, k)) return SHERRY_E_SHAPE;
  const int64_t R = ceil_div(n, kTileRows);
  const int C = static_cast<int>(ceil_div(k, kTileK));
  const int S = (R * gemv_split(C) >= 4096) ? gemv_split(C) : kGemvWaves;
  const dim3 grid(static_cast<unsigned>(ceil_div(R * S, kGemvWaves)));
  const dim3 block(kGemvThreads);
  if (gs) {
    switch (m) {
      case 1: return launch(gemv_tok_kernel<1, true>, grid, block, 0, s, w, x, x_scale, ws, gs, y, acc, n, k, S);
      case 2: return launch(gemv_tok_kernel<2, true>, grid, block, 0, s, w, x, x_scale, ws, gs, y, acc, n, k, S);
      case 3: return launch(gemv_tok_kernel<3, true>, grid, block, 0, s, w, x, x_scale, ws, gs, y, acc, n, k, S);
      default: return launch(gemv_tok_kernel<4, true>, grid, block, 0, s, w, x, x_scale, ws, gs, y, acc, n, k, S);
    }
  }
  switch (m) {
    case 1: return launch(gemv_tok_kernel<1, false>, grid, block, 0, s, w, x, x_scale, ws, gs, y, acc, n, k, S);
    case 2: return launch(gemv_tok_kernel<2, false>, grid, block, 0, s, w, x, x_scale, ws, gs, y, acc, n, k, S);
    case 3: return launch(gemv_tok_kernel<3, false>, grid, block, 0, s, w, x, x_scale, ws, gs, y, acc, n, k, S);
    default: return launch(gemv_tok_kernel<4, false>, grid, block, 0, s, w, x, x_scale, ws, gs, y, acc, n, k, S);
  }
}

int64_t gemv_tok_blocks(int64_t n, int64_t k) {
  return ceil_div(ceil_div(n, kTileRows) * gemv_split(static_cast<int>(ceil_div(k, kTileK))),
                  kGemvWaves);
}

int launch_gemv_tok_il_batched(const sherry_gemm_desc* descs, int count, int64_t total_blocks,
                               hipStream_t s) {
  return launch(gemv_tok_il_batched_kernel, dim3(static_cast<unsigned>(total_blocks)),
                dim3(kGemvThreads), 0, s, descs, count);
}

int launch_gemv_tok_batched(const sherry_gemm_desc* descs, int count, int64_t total_blocks,
                            bool groups, hipStream_t s) {
  if (groups)
    return launch(gemv_tok_batched_kernel<true>, dim3(static_cast<unsigned>(total_blocks)),
                  dim3(kGemvThreads), 0, s, descs, count);
  return launch(gemv_tok_batched_kernel<false>, dim3(static_cast<unsigned>(total_blocks)),
                dim3(kGemvThreads), 0, s, descs, count);
}

int launch_gemv_group(const uint8_t* w, const int8_t* x, const float* x_scale, const float* gs,
                      float* y, int32_t* acc, int64_t m, int64_t n, int64_t k, hipStream_t s) {
  const int64_t R = ceil_div(n, kTileRows);
  const int C = static_cast<int>(ceil_div(k, kTileK));
  const int S = (R * gemv_split(C) >= 4096) ? gemv_split(C) : kGemvWaves;
  const dim3 grid(static_cast<unsigned>(ceil_div(R * S, kGemvWaves)));
  const dim3 block(kGemvThreads);
  switch (m) {
    case 1: return launch(gemv_group_kernel<1>, grid, block, 0, s, w, x, x_scale, gs, y, acc, n, k, S);
    case 2: return launch(gemv_group_kernel<2>, grid, block, 0, s, w, x, x_scale, gs, y, acc, n, k, S);
    case 3: return launch(gemv_group_kernel<3>, grid, block, 0, s, w, x, x_scale, gs, y, acc, n, k, S);
    case 4: return launch(gemv_group_kernel<4>, grid, block, 0, s, w, x, x_scale, gs, y, acc, n, k, S);
    default: return SHERRY_E_SHAPE;
  }
}

int launch_gemv_f32_group(const uint8_t* w, const float* x, float* x_scale, const float* gs,
                          float* y, int32_t* acc, int64_t n, int64_t k, hipStream_t s) {
  const int64_t R = ceil_div(n, kTileRows);
  const int C = static_cast<int>(ceil_div(k, kTileK));
  const int S = (R * gemv_split(C, kFusedTarget) >= 4096) ? gemv_split(C, kFusedTarget) : kGemvWaves;
  return launch(gemv_f32_group_kernel, dim3(static_cast<unsigned>(ceil_div(R * S, kGemvWaves))),
                dim3(kGemvThreads), 0, s, w, x, x_scale, gs, y, acc, n, k, S);
}

int launch_gemv_batched(const sherry_gemv_desc* descs, int count, int64_t total_blocks,
                        hipStream_t s) {
  return launch(gemv_batched_kernel, dim3(static_cast<unsigned>(total_blocks)),
                dim3(kGemvThreads), 0, s, descs, count);
}

int launch_gemv_f32(const uint8_t* w, const float* x, float* x_scale, WScale ws, float* y,
                    int32_t* acc, int64_t n, int64_t k, hipStream_t s) {
  const int64_t R = ceil_div(n, kTileRows);
  const int C = static_cast<int>(ceil_div(k, kTileK));
  const int S = (R * gemv_split(C, kFusedTarget) >= 4096) ? gemv_split(C, kFusedTarget) : kGemvWaves;
  return launch(gemv_f32_kernel, dim3(static_cast<unsigned>(ceil_div(R * S, kGemvWaves))),
                dim3(kGemvThreads), 0, s, w, x, x_scale, ws, y, acc, n, k, S);
}

int launch_gemv_f32_batched(const sherry_gemv_f32_desc* descs, int count, int64_t total_blocks,
                            bool il, hipStream_t s) {
  if (il)
    return launch(gemv_f32_batched_kernel<true>, dim3(static_cast<unsigned>(total_blocks)),
                  dim3(kGemvThreads), 0, s, descs, count);
  return launch(gemv_f32_batched_kernel<false>, dim3(static_cast<unsigned>(total_blocks)),
                dim3(kGemvThreads), 0, s, descs, count);
}

}  // namespace sherry
