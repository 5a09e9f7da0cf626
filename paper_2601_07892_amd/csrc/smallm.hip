// Products of up to 16 tokens on the matrix cores, with the weights in the
// registers they are loaded into (Eq. 2; grouped launches of small-M decode
// steps).
//
// Work mapping.  A workgroup is 4 waves; wave w owns 64-row tile 4g + w and
// the whole K of it (lane i = row i, as in the decode GEMV), streaming its
// units through a register ring and decoding each code through the 32-entry
// LDS table.  The 4 waves walk K in lockstep windows of kWinUnits units: the
// activations of a window (16 token rows x 1024 K values, int8) are staged in
// LDS by the whole workgroup, double-buffered, one window ahead.  (Four
// waves per workgroup rather than eight: twice the workgroups to balance the
// chip and half the waves held at each window barrier; 4% faster on a 3B
// step of 16 tokens.)
//
// Every global load is issued on every path (past the end of a tile or of k
// it reads zeros through an empty or bounded resource), so the compiler's
// waits count exact numbers of loads instead of draining the queue; a
// drained queue before each unit cost a quarter of the throughput.
//
// Operands.  v_mfma_i32_32x32x32_i8 takes B[k][j] from lane j + 32h (k half
// h) and A[i][k] from lane i + 32h.  The four looked-up words of a 4-code
// chunk are B as they stand: lanes 0-31 give k half 0 = rows 0-31 of the
// tile, lanes 32-63 give k half 1 = rows 32-63, both over the same 16
// activations.  A row m (k half 0, lane m) and A row 16 + m (k half 1, lane
// 48 + m) carry token m's 16 activations of the chunk; every other lane's A
// stays zero.  So D[m][t] = x_m . w(row t) and D[16 + m][t] = x_m . w(row
// 32 + t): one MFMA per chunk serves 64 rows and 16 tokens, with no lane
// exchange of the weights.
//
// On lane-interleaved units (kIL) each 4-code chunk slot of a lane is the B
// operand of a v_mfma_i32_16x16x64_i8 over 16 rows and 64 weights instead;
// lane 16b + m reads token m's chunks b and 4 + b of the unit from the
// stage, an A operand that serves all four row groups (two 16-byte LDS reads
// per unit and lane), and D[m][t] of row group g lands in lane 16(m/4) + t.
#include "sherry_internal.h"

namespace sherry {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));

constexpr int kSmWaves = 4;
constexpr int kSmThreads = 64 * kSmWaves;
constexpr int kSmTok = 16;                      // token rows staged
constexpr int kWinUnits = 8;                    // units per window
constexpr int kWinK = kWinUnits * kTileK;       // 1024 K values
constexpr int kRowStride = kWinK + 16;          // staged token row, padded
constexpr int kStageBytes = kSmTok * kRowStride;
constexpr int kWinPieces = kSmTok * kWinK / 16 / kSmThreads;  // 16-byte pieces per thread
constexpr int kSmRing = 4;                      // units per wave in the register ring
static_assert(kWinUnits % kSmRing == 0, "ring slots repeat in every window");

// Table lookups of codes j0 .. j0 + 15 of a unit row (lane i = row i):
// wv[j] = the int8x4 weights of code j0 + j.
template <int j0, int... js>
__device__ __forceinline__ void sm_lookup(const uint32_t (&d)[5], const uint32_t* lut,
                                          uint32_t (&wv)[16], std::integer_sequence<int, js...>) {
  ((wv[js] = *reinterpret_cast<const uint32_t*>(reinterpret_cast<const char*>(lut) +
                                                code_x4<j0 + js>(d))),
   ...);
}

// Stage layout: token row t at t * kRowStride, its 16-byte piece p (K offset
// 16p in the window) at 16p within it; the 16-byte pad per row puts the
// lanes that read one piece of consecutive rows on different 4-bank groups.
__device__ __forceinline__ int stage_off(int t, int p) { return t * kRowStride + 16 * p; }

// The window's activations for this thread: piece i * kSmThreads + tid of the
// window, i.e. token row q / 64, piece q % 64, read through a resource over
// the m x k activations (rows past m read zeros).  Pieces are 16-byte loads
// when k % 16 == 0 (the activations are 16-byte aligned), else four word
// loads (k % 4 == 0).  A piece or word at or past k is loaded from an offset
// outside the resource, so it reads zeros without touching memory and no
// load reaches into the next row; every load is issued on every path.
constexpr int kSmOutside = 0x40000000;  // past any m * k (m <= 16, k <= 2^18)

__device__ __forceinline__ void stage_load(u32x4 (&v)[kWinPieces], __amdgpu_buffer_rsrc_t rx,
                                           int k, int w) {
  const bool wide = (k & 15) == 0;
#pragma unroll
  for (int i = 0; i < kWinPieces; ++i) {
    const int q = i * kSmThreads + static_cast<int>(threadIdx.x);
    const int t = q / (kWinK / 16), p = q % (kWinK / 16);
    const int kk = w * kWinK + 16 * p;  // first K value of the piece
    const int left = k - kk;            // K values of the row left from kk
    const int off = t * k + kk;
    if (wide) {
      v[i] = __builtin_amdgcn_raw_buffer_load_b128(rx, left >= 16 ? off : kSmOutside, 0, 0);
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e)
        v[i][e] = __builtin_amdgcn_raw_buffer_load_b32(rx, 4 * e < left ? off + 4 * e : kSmOutside,
                                                       0, 0);
    }
  }
}

__device__ __forceinline__ void stage_store(const u32x4 (&v)[kWinPieces], int8_t* st) {
#pragma unroll
  for (int i = 0; i < kWinPieces; ++i) {
    const int q = i * kSmThreads + static_cast<int>(threadIdx.x);
    const int t = q / (kWinK / 16), p = q % (kWinK / 16);
    *reinterpret_cast<u32x4*>(st + stage_off(t, p)) = v[i];
  }
}

// Barrier for LDS traffic only: outstanding global loads stay in flight.
__device__ __forceinline__ void sm_lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

struct SmProblem {
  const uint8_t* w;
  const int8_t* x;
  const float* x_scale;
  float* y;
  int32_t* acc;
  int n, k, m;
  WScale ws;
  const float* gs;  // per-group scales [n][k/128], or nullptr
};

// One workgroup: tiles kSmWaves*g .. kSmWaves*g + kSmWaves - 1 of the
// problem.  lds: the table (128 bytes), two stages, a zero row (the A
// operand of lanes that carry no token, read like a token row so that no
// lane branches) and the tokens' activation scales.
//
// kG: per-group scales (one per row and unit; k % 512 == 0 and p.gs 16-byte
// aligned, so that a lane reads four units' scales of its row at once).
// Each unit's MFMAs then run as one chain from zero into c[u & 1], and the
// unit is scaled one unit later (its chain has completed by then) into fp32
// accumulators: element e < 8 of a lane belongs to row l % 32 of the tile,
// e >= 8 to row l % 32 + 32, whose scales a lane-half swap of the loaded
// ones provides.
//
// kIL: lane-interleaved weights (sherry_pack_il; not with kG).  Lane 16b + t
// holds, as chunk slot (g, p), row 16g + t's weights of chunk 4p + b, the B
// operand of one v_mfma_i32_16x16x64_i8 over 16 rows and 64 weights; its A
// operand, token m = lane % 16's chunks b and 4 + b of the unit, is read once
// per unit and serves the four row groups.  D[m][t] lands in lane
// 16(m/4) + t, element m % 4 of accumulator g.
template <bool kG, bool kIL = false>
__device__ __forceinline__ void sm_block(const SmProblem& p, int g, uint32_t* lut,
                                         int8_t* stages, int8_t* zrow, float* xs) {
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int C = (p.k + kTileK - 1) / kTileK;
  const int R = (p.n + kTileRows - 1) / kTileRows;
  const int r = g * kSmWaves + wave;
  const bool live = r < R;
  // this wave's tile (dead waves: no units)
  const UnitRun tile{p.w + int64_t(live ? r : 0) * C * kUnitBytes, live ? C : 0};
  const __amdgpu_buffer_rsrc_t rx = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<int8_t*>(p.x), 0, p.m * p.k, kBufferWord3);
  const int nwin = (C + kWinUnits - 1) / kWinUnits;

  // token of this lane's A operand (lanes 0-15 and 48-63; staged rows past m
  // are zero), or none
  const int tok = lane < 16 ? lane : (lane >= 48 ? lane - 48 : -1);

  // the scales and window 0 first, then the ring: the stage store waits for
  // the former only
  float xsv = 0.0f;
  if (tid < p.m) xsv = as_global(p.x_scale)[tid];
  u32x4 sv[kWinPieces];
  stage_load(sv, rx, p.k, 0);
  __builtin_amdgcn_sched_barrier(0);
  uint32_t ring[kSmRing][5];
#pragma unroll
  for (int u = 0; u < kSmRing; ++u) {
    load_unit(ring[u], tile, u, lane);
    __builtin_amdgcn_sched_barrier(0);
  }
  if (tid < 32) lut[tid] = decode_word(tid);
  if (tid < kWinK / 16) reinterpret_cast<u32x4*>(zrow)[tid] = u32x4{0u, 0u, 0u, 0u};
  if (tid < kSmTok) xs[tid] = xsv;
  stage_store(sv, stages);
  sm_lds_barrier();  // window 0, the table, the zero row and the scales are ready

  // per-group scales: lane l reads row l of the tile, four units per load,
  // two chunks ahead; slo / shi hold the current chunk's scales of rows
  // l % 32 and l % 32 + 32, plo / phi the previous chunk's last ones
  const int grows =
      kG && live ? (p.n - r * kTileRows < kTileRows ? p.n - r * kTileRows : kTileRows) : 0;
  const __amdgpu_buffer_rsrc_t gr = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<float*>(p.gs) + int64_t(live ? r : 0) * kTileRows * C, 0, grows * C * 4,
      kBufferWord3);
  u32x4 gqa{}, gqb{};
  float slo[4] = {}, shi[4] = {}, plo = 0.0f, phi = 0.0f;
  float accf[16] = {};
  if constexpr (kG) {
    gqa = __builtin_amdgcn_raw_buffer_load_b128(gr, 4 * (lane * C), 0, 0);
    gqb = __builtin_amdgcn_raw_buffer_load_b128(gr, 4 * (lane * C + 4), 0, 0);
  }

  static_assert(!(kG && kIL), "per-group scales: tiled units only");
  v16i c[2] = {v16i{}, v16i{}};
  v4i acc4[4] = {};  // kIL accumulators, one per row group
  for (int w = 0; w < nwin; ++w) {
    // the next window's activations are in flight during this one
    stage_load(sv, rx, p.k, w + 1);
    // this lane's A row of the window
    const int8_t* arow =
        tok >= 0 ? stages + (w & 1) * kStageBytes + tok * kRowStride : zrow;
#pragma unroll
    for (int u = 0; u < kWinUnits; ++u) {
      const int j = w * kWinUnits + u;  // unit of the tile
      if constexpr (kG) {
        if (u % 4 == 0) {  // a new chunk of four units (issued on every path)
          plo = slo[3];
          phi = shi[3];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const uint32_t own = gqa[e];
            const auto sw = __builtin_amdgcn_permlane32_swap(own, own, false, false);
            slo[e] = __uint_as_float(sw[0]);
            shi[e] = __uint_as_float(sw[1]);
          }
          gqa = gqb;
          gqb = __builtin_amdgcn_raw_buffer_load_b128(gr, 4 * (lane * C + j + 8), 0, 0);
        }
      }
      if (kIL && j < C) {
        // the unit's activation operands: token lane % 16 (rows past m are
        // zero in the stage), chunks b and 4 + b, b = lane / 16
        const int8_t* ar = stages + (w & 1) * kStageBytes + (lane & 15) * kRowStride +
                           16 * (8 * u + (lane >> 4));
        const v4i xa[2] = {*reinterpret_cast<const v4i*>(ar),
                           *reinterpret_cast<const v4i*>(ar + 64)};
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          __builtin_amdgcn_sched_barrier(0);
          uint32_t wv[16];
          if (h == 0) sm_lookup<0>(ring[u % kSmRing], lut, wv, std::make_integer_sequence<int, 16>{});
          else sm_lookup<16>(ring[u % kSmRing], lut, wv, std::make_integer_sequence<int, 16>{});
          // slots (g, p) = (2h + (s >> 1), s & 1), alternating accumulators
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int sl = (i & 1) * 2 + (i >> 1);  // 0, 2, 1, 3
            const v4i b = {static_cast<int>(wv[4 * sl]), static_cast<int>(wv[4 * sl + 1]),
                           static_cast<int>(wv[4 * sl + 2]), static_cast<int>(wv[4 * sl + 3])};
            acc4[2 * h + (sl >> 1)] =
                __builtin_amdgcn_mfma_i32_16x16x64_i8(xa[sl & 1], b, acc4[2 * h + (sl >> 1)], 0, 0, 0);
          }
        }
      } else if (j < C) {
        // codes 16h .. 16h + 15: 16 table reads in flight, then 4 chunks
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          __builtin_amdgcn_sched_barrier(0);
          uint32_t wv[16];
          if (h == 0) sm_lookup<0>(ring[u % kSmRing], lut, wv, std::make_integer_sequence<int, 16>{});
          else sm_lookup<16>(ring[u % kSmRing], lut, wv, std::make_integer_sequence<int, 16>{});
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const v4i a = *reinterpret_cast<const v4i*>(arow + 16 * (8 * u + 4 * h + q));
            const v4i b = {static_cast<int>(wv[4 * q]), static_cast<int>(wv[4 * q + 1]),
                           static_cast<int>(wv[4 * q + 2]), static_cast<int>(wv[4 * q + 3])};
            if constexpr (kG) {
              const v16i cin = (h == 0 && q == 0) ? v16i{} : c[u & 1];
              c[u & 1] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a, b, cin, 0, 0, 0);
            } else {
              c[q & 1] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a, b, c[q & 1], 0, 0, 0);
            }
          }
        }
      }
      if constexpr (kG) {
        if (j >= 1 && j <= C) {  // unit j - 1, in c[(u + 1) & 1]
          const float sl = (u % 4 == 0) ? plo : slo[(u + 3) % 4];
          const float sh = (u % 4 == 0) ? phi : shi[(u + 3) % 4];
#pragma unroll
          for (int e = 0; e < 16; ++e)
            accf[e] = __builtin_fmaf(static_cast<float>(c[(u + 1) & 1][e]), e < 8 ? sl : sh,
                                     accf[e]);
        }
      }
      __builtin_amdgcn_sched_barrier(0);
      load_unit(ring[u % kSmRing], tile, j + kSmRing, lane);
      __builtin_amdgcn_sched_barrier(0);
    }
    stage_store(sv, stages + ((w + 1) & 1) * kStageBytes);
    sm_lds_barrier();
  }

  if constexpr (kG) {
    // the last unit (C % 8 == 0: the walk ended on it), in c[1]
    if (C % kWinUnits == 0) {
#pragma unroll
      for (int e = 0; e < 16; ++e)
        accf[e] = __builtin_fmaf(static_cast<float>(c[1][e]), e < 8 ? slo[3] : shi[3], accf[e]);
    }
  }

  // epilogue: lane l, element e holds D[i][l % 32] with i = 8(e/4) + 4(l/32)
  // + e%4: token i % 16 of tile row (l % 32) + 32 (i / 16).  The scales are
  // fetched once (two rows per lane), then every element is stored.
  if (!live) return;
  if constexpr (kG) {
    __builtin_amdgcn_s_waitcnt(0);
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int i = 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
      const int t = i & 15;
      const int64_t row = int64_t(r) * kTileRows + (lane & 31) + 32 * (i >> 4);
      if (t < p.m && row < p.n) as_global_mut(p.y)[int64_t(t) * p.n + row] = accf[e] * xs[t];
    }
    return;
  }
  if constexpr (kIL) {
    // lane l, accumulator g, element e: token 4(l / 16) + e of tile row
    // 16g + l % 16
    float wsg[4];
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int64_t row = int64_t(r) * kTileRows + 16 * g + (lane & 15);
      wsg[g] = p.ws.at(row < p.n ? row : p.n - 1);
    }
    __builtin_amdgcn_s_waitcnt(0);
#pragma unroll
    for (int g = 0; g < 4; ++g) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int t = 4 * (lane >> 4) + e;
        const int64_t row = int64_t(r) * kTileRows + 16 * g + (lane & 15);
        const int32_t v = acc4[g][e];
        const float sc = xs[t] * wsg[g];
        if (t < p.m && row < p.n) {
          as_global_mut(p.y)[int64_t(t) * p.n + row] = static_cast<float>(v) * sc;
          if (p.acc) as_global_mut(p.acc)[int64_t(t) * p.n + row] = v;
        }
      }
    }
    return;
  }
  const int64_t row0 = int64_t(r) * kTileRows + (lane & 31);
  const float ws0 = p.ws.at(row0 < p.n ? row0 : p.n - 1);
  const float ws1 = p.ws.at(row0 + 32 < p.n ? row0 + 32 : p.n - 1);
  // one wait for every load of the wave (the scales; the ring is drained),
  // so that no store below waits for the stores before it
  __builtin_amdgcn_s_waitcnt(0);
#pragma unroll
  for (int e = 0; e < 16; ++e) {
    const int i = 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
    const int t = i & 15;
    const int64_t row = row0 + 32 * (i >> 4);
    const int32_t v = c[0][e] + c[1][e];
    const float s = xs[t] * ((i >> 4) ? ws1 : ws0);
    if (t < p.m && row < p.n) {
      as_global_mut(p.y)[int64_t(t) * p.n + row] = static_cast<float>(v) * s;
      if (p.acc) as_global_mut(p.acc)[int64_t(t) * p.n + row] = v;
    }
  }
}

// kGroups: some descriptor carries per-group scales (a kernel of its own,
// so that the other keeps its registers).
template <bool kGroups>
__global__ __launch_bounds__(kSmThreads) __attribute__((amdgpu_waves_per_eu(kGroups ? 3 : 4))) void smallm_batched_kernel(
    const sherry_gemm_desc* __restrict__ descs, int count) {
  __shared__ uint32_t lut[32];
  __shared__ __attribute__((aligned(16))) int8_t stages[2 * kStageBytes];
  __shared__ __attribute__((aligned(16))) int8_t zrow[kWinK];
  __shared__ float xs[kSmTok];
  const int32_t blk = static_cast<int32_t>(blockIdx.x);
  const int lo = find_block_desc(descs, count, blk);
  if (lo < 0) return;
  const sherry_gemm_desc& d = descs[lo];
  const SmProblem p{d.w, d.x, d.x_scale, d.y, d.acc, d.n, d.k, d.m,
                    WScale{d.w_scales, d.w_scale}, d.w_group_scales};
  if (kGroups && p.gs) sm_block<kGroups>(p, blk - d.block_begin, lut, stages, zrow, xs);
  else sm_block<false>(p, blk - d.block_begin, lut, stages, zrow, xs);
}

// Grouped products of up to 16 tokens on lane-interleaved weights.
__global__ __launch_bounds__(kSmThreads) __attribute__((amdgpu_waves_per_eu(4))) void smallm_il_batched_kernel(
    const sherry_gemm_desc* __restrict__ descs, int count) {
  __shared__ uint32_t lut[32];
  __shared__ __attribute__((aligned(16))) int8_t stages[2 * kStageBytes];
  __shared__ __attribute__((aligned(16))) int8_t zrow[kWinK];
  __shared__ float xs[kSmTok];
  const int32_t blk = static_cast<int32_t>(blockIdx.x);
  const int lo = find_block_desc(descs, count, blk);
  if (lo < 0) return;
  const sherry_gemm_desc& d = descs[lo];
  const SmProblem p{d.w, d.x, d.x_scale, d.y, d.acc, d.n, d.k, d.m,
                    WScale{d.w_scales, d.w_scale}, nullptr};
  sm_block<false, true>(p, blk - d.block_begin, lut, stages, zrow, xs);
}

}  // namespace

int launch_smallm_il_batched(const sherry_gemm_desc* descs, int count, int64_t total_blocks,
                             hipStream_t s) {
  return launch(smallm_il_batched_kernel, dim3(static_cast<unsigned>(total_blocks)),
                dim3(kSmThreads), 0, s, descs, count);
}

int64_t smallm_blocks(int64_t n) { return ceil_div(ceil_div(n, kTileRows), kSmWaves); }

int launch_smallm_batched(const sherry_gemm_desc* descs, int count, int64_t total_blocks,
                          bool groups, hipStream_t s) {
  if (groups)
    return launch(smallm_batched_kernel<true>, dim3(static_cast<unsigned>(total_blocks)),
                  dim3(kSmThreads), 0, s, descs, count);
  return launch(smallm_batched_kernel<false>, dim3(static_cast<unsigned>(total_blocks)),
                dim3(kSmThreads), 0, s, descs, count);
}

}  // namespace sherry
