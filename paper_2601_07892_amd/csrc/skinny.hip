// Small-M product (a few to 64 tokens; Eq. 2): the weight stream of the
// decode kernel, with the multiply-accumulate on int8 MFMA.
//
// Work mapping.  A workgroup is 8 waves; wave w owns 64-row tile 8*g + w and
// streams all of its containers in order (no split along K, so no partial
// sums to combine).  The waves walk K in lockstep chunks: the activations of
// chunk ch (all tokens, kSkChunk/MT values each) sit in one of two LDS
// stages while the next chunk is loaded into registers.
//
// Per container (64 rows x 128 weights) a wave decodes its 32 codes per lane
// through the 32-entry table (lane i = row i), exactly as the decode kernel
// does.  v_permlane32_swap then pairs rows i and i + 32 so that each 16-byte
// operand holds one row group's weights in the MFMA layout (lane l: row
// l%32, k half l/32), and v_mfma_i32_32x32x32_i8 accumulates
// C[token][row] for 32 tokens x 32 rows per instruction: 8 MFMAs per
// container and 32-token block.
#include "sherry_internal.h"

namespace sherry {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));

constexpr int kSkWaves = 8;
constexpr int kSkThreads = 64 * kSkWaves;
constexpr int kSkRing = 4;        // containers per wave in the register ring
constexpr int kSkLutBytes = 128;  // the code table, at LDS address 0
// K values per staged chunk and token block count: MT blocks of 32 tokens
// share 32 KB per stage (chunk = 1024 / MT values, a multiple of the ring)
template <int MT>
struct SkCfg {
  static constexpr int TOK = 32 * MT;             // staged token rows
  static constexpr int KC = 1024 / MT;            // K values per chunk
  static constexpr int ROW = KC + 16;             // LDS row stride (bank skew)
  static constexpr int UPC = KC / kTileK;         // containers per chunk
  static constexpr int STAGE = TOK * ROW;
  static constexpr int SPT = TOK * KC / 16 / kSkThreads;  // 16-byte pieces per thread
  static_assert(UPC % kSkRing == 0, "chunks hold whole ring turns");
  static_assert(SPT * 16 * kSkThreads == TOK * KC, "stage split");
};

// One product of a batch (or the whole single-product launch).
struct SkProblem {
  const uint8_t* w;
  const int8_t* x;
  const float* x_scale;
  float* y;
  int32_t* acc;
  int n, k, m;
  float w_scale;
};

__device__ __forceinline__ void sk_load_container(uint32_t (&d)[5], __amdgpu_buffer_rsrc_t r,
                                                  int c, int lane) {
  const u32x4 h =
      __builtin_amdgcn_raw_buffer_load_b128(r, 16 * lane, c * kUnitBytes, kLoadStream);
  d[0] = h.x;
  d[1] = h.y;
  d[2] = h.z;
  d[3] = h.w;
  d[4] = __builtin_amdgcn_raw_buffer_load_b32(r, kHeadBytes + 4 * lane, c * kUnitBytes,
                                              kLoadStream);
}

template <int j0, int... js>
__device__ __forceinline__ void sk_offsets(const uint32_t (&d)[5], uint32_t* a4,
                                           std::integer_sequence<int, js...>) {
  ((a4[js] = code_x4<j0 + js>(d)), ...);
}

// Decodes container d and accumulates its 128 K values against the staged
// activations xb (row stride ROW, K offset koff) into c[row group][token block].
template <int MT>
__device__ __forceinline__ void sk_container(const uint32_t (&d)[5], const int8_t* xb,
                                             int koff, const uint32_t* lut,
                                             v16i (&c)[2][MT]) {
  using G = SkCfg<MT>;
  const int lane = threadIdx.x & 63;
  uint32_t a4[32];
  sk_offsets<0>(d, a4, std::make_integer_sequence<int, 32>{});
  uint32_t wv[32];
#pragma unroll
  for (int j = 0; j < 32; ++j)
    wv[j] = *reinterpret_cast<const uint32_t*>(reinterpret_cast<const char*>(lut) + a4[j]);
  const int8_t* xl = xb + (lane & 31) * G::ROW + koff + 16 * (lane >> 5);
#pragma unroll
  for (int s = 0; s < 4; ++s) {
    // words 8s..8s+3 hold K 32s..32s+15 of this lane's row, 8s+4..8s+7 the
    // next 16; after the swap lo = rows 0-31 and hi = rows 32-63 in the
    // operand layout
    v4i lo, hi;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const auto r = __builtin_amdgcn_permlane32_swap(wv[8 * s + i], wv[8 * s + 4 + i], false,
                                                      false);
      lo[i] = static_cast<int>(r[0]);
      hi[i] = static_cast<int>(r[1]);
    }
#pragma unroll
    for (int tb = 0; tb < MT; ++tb) {
      const v4i xv = *reinterpret_cast<const v4i*>(xl + tb * 32 * G::ROW + 32 * s);
      c[0][tb] = __builtin_amdgcn_mfma_i32_32x32x32_i8(xv, lo, c[0][tb], 0, 0, 0);
      c[1][tb] = __builtin_amdgcn_mfma_i32_32x32x32_i8(xv, hi, c[1][tb], 0, 0, 0);
    }
  }
}

// Barrier for LDS traffic only (outstanding global loads stay in flight).
__device__ __forceinline__ void sk_lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Workgroup g of problem p: tiles T*g .. T*g+T-1 (T = 8/S), each split along
// K over S waves (wave w: tile w/S, split w%S).  Split s owns units
// [s*U, min((s+1)*U, C)) with U = ceil(C/S); all waves walk their ranges in
// lockstep chunks of UPC_S = UPC/S units, and a stage holds, for every
// token, the S splits' windows side by side.  With S > 1 the partial
// accumulators meet in LDS (over the stages) and split 0 writes the tile.
template <int MT, int S>
__device__ __forceinline__ void sk_block(const SkProblem& p, int g, const uint32_t* lut,
                                         int8_t* xs) {
  using G = SkCfg<MT>;
  static_assert(S >= 1 && G::UPC % S == 0, "splits divide a chunk");
  constexpr int T = kSkWaves / S;   // tiles per workgroup
  constexpr int UPS = G::UPC / S;   // units per split per chunk
  constexpr int WIN = UPS * kTileK; // K values per split window
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int C = (p.k + kTileK - 1) / kTileK;
  const int R = (p.n + kTileRows - 1) / kTileRows;
  const int U = (C + S - 1) / S;    // units per split
  const int r = g * T + wave / S;
  const int sp = wave % S;
  const int u0 = sp * U, u1 = (u0 + U < C) ? u0 + U : C;
  const bool live = r < R && u0 < u1;
  const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(p.w) + (int64_t(r < R ? r : 0) * C + (live ? u0 : 0)) * kUnitBytes, 0,
      live ? (u1 - u0) * kUnitBytes : 0, kBufferWord3);
  const int nch = (U + UPS - 1) / UPS;
  const bool k16 = (p.k & 15) == 0;

  // activation chunk ch -> registers: piece q = tid + threads*v is token
  // q / (KC/16), 16 bytes at window offset 16 * (q % (KC/16)): split
  // window s = offset / WIN, K = (s*U + ch*UPS)*128 + offset % WIN; zero past
  // m, past k and past the split's end
  uint4 sv[G::SPT];
  auto stage_load = [&](int ch) {
#pragma unroll
    for (int v = 0; v < G::SPT; ++v) {
      const int q = tid + kSkThreads * v;
      const int tok = q / (G::KC / 16), o = 16 * (q % (G::KC / 16));
      const int ws = o / WIN, wo = o % WIN;
      const int ub = ws * U + ch * UPS;  // first unit of this window
      const int kk = ub * kTileK + wo;
      const int kend = (ws * U + U < C ? ws * U + U : C) * kTileK;
      uint4 val = make_uint4(0, 0, 0, 0);
      if (tok < p.m && kk < p.k && kk < kend) {
        const int8_t* src = p.x + int64_t(tok) * p.k + kk;
        if (k16) {
          val = *reinterpret_cast<const uint4*>(as_global(src));
        } else {
          uint32_t t4[4] = {0, 0, 0, 0};
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (kk + 4 * e < p.k) t4[e] = *reinterpret_cast<const uint32_t*>(as_global(src + 4 * e));
          val = make_uint4(t4[0], t4[1], t4[2], t4[3]);
        }
      }
      sv[v] = val;
    }
  };
  auto stage_store = [&](int buf) {
#pragma unroll
    for (int v = 0; v < G::SPT; ++v) {
      const int q = tid + kSkThreads * v;
      const int tok = q / (G::KC / 16), kc = q % (G::KC / 16);
      *reinterpret_cast<uint4*>(xs + buf * G::STAGE + tok * G::ROW + 16 * kc) = sv[v];
    }
  };

  v16i c[2][MT];
#pragma unroll
  for (int h = 0; h < 2; ++h)
#pragma unroll
    for (int tb = 0; tb < MT; ++tb) c[h][tb] = v16i{};

  stage_load(0);
  stage_store(0);
  if (nch > 1) stage_load(1);
  uint32_t ring[kSkRing][5];
#pragma unroll
  for (int u = 0; u < kSkRing; ++u) {
    sk_load_container(ring[u], rs, u, lane);
    __builtin_amdgcn_sched_barrier(0);
  }
  sk_lds_barrier();  // stage 0 and the table are ready

  // unit j of the split (relative to u0) lives in chunk j / UPS; at each
  // chunk boundary the next stage (in registers) is written and the one
  // after it is loaded
  const int nunits = nch * UPS;
  for (int j = 0; j < nunits; j += kSkRing) {
#pragma unroll
    for (int u = 0; u < kSkRing; ++u) {
      const int jj = j + u;
      const int ch = jj / UPS;
      if (jj % UPS == 0 && jj > 0) {
        stage_store(ch & 1);
        sk_lds_barrier();
        if (ch + 1 < nch) stage_load(ch + 1);
      }
      const int8_t* xb = xs + (ch & 1) * G::STAGE + sp * WIN;
      if (live && u0 + jj < u1) sk_container<MT>(ring[u], xb, (jj % UPS) * kTileK, lut, c);
      __builtin_amdgcn_sched_barrier(0);
      sk_load_container(ring[u], rs, jj + kSkRing, lane);
      __builtin_amdgcn_sched_barrier(0);
    }
  }

  if constexpr (S > 1) {
    // partial sums of the S splits of a tile through LDS (the stages are
    // free now), one token block at a time: [wave][h][element][lane]
    int32_t* red = reinterpret_cast<int32_t*>(xs);
    static_assert(kSkWaves * 2 * 16 * 64 * 4 <= 2 * G::STAGE, "reduction fits the stages");
#pragma unroll
    for (int tb = 0; tb < MT; ++tb) {
      sk_lds_barrier();
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int e = 0; e < 16; ++e) red[((wave * 2 + h) * 16 + e) * 64 + lane] = c[h][tb][e];
      sk_lds_barrier();
      if (sp == 0) {
#pragma unroll
        for (int q = 1; q < S; ++q)
#pragma unroll
          for (int h = 0; h < 2; ++h)
#pragma unroll
            for (int e = 0; e < 16; ++e)
              c[h][tb][e] += red[(((wave + q) * 2 + h) * 16 + e) * 64 + lane];
      }
    }
  }

  // epilogue (split 0 of each tile): lane holds C[token][row] for row =
  // 32h + lane%32 of the tile and token = 32tb + 8(e/4) + 4(lane/32) + e%4,
  // e = accumulator element
  if (r >= R || sp != 0) return;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int row = r * kTileRows + 32 * h + (lane & 31);
    if (row >= p.n) continue;
#pragma unroll
    for (int tb = 0; tb < MT; ++tb) {
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int tok = 32 * tb + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
        if (tok >= p.m) continue;
        const int32_t v = c[h][tb][e];
        const float s = as_global(p.x_scale)[tok] * p.w_scale;
        as_global_mut(p.y)[int64_t(tok) * p.n + row] = static_cast<float>(v) * s;
        if (p.acc) as_global_mut(p.acc)[int64_t(tok) * p.n + row] = v;
      }
    }
  }
}

template <int MT, int S>
__global__ __launch_bounds__(kSkThreads) void skinny_kernel(SkProblem p) {
  __shared__ __attribute__((aligned(16))) int8_t lds[kSkLutBytes + 2 * SkCfg<MT>::STAGE];
  uint32_t* lut = reinterpret_cast<uint32_t*>(lds);
  if (threadIdx.x < 32) lut[threadIdx.x] = decode_word(threadIdx.x);
  sk_block<MT, S>(p, blockIdx.x, lut, lds + kSkLutBytes);
}

template <int MT>
__global__ __launch_bounds__(kSkThreads) void skinny_batched_kernel(
    const sherry_gemm_desc* __restrict__ descs, int count) {
  __shared__ __attribute__((aligned(16))) int8_t lds[kSkLutBytes + 2 * SkCfg<MT>::STAGE];
  uint32_t* lut = reinterpret_cast<uint32_t*>(lds);
  if (threadIdx.x < 32) lut[threadIdx.x] = decode_word(threadIdx.x);
  const int32_t blk = static_cast<int32_t>(blockIdx.x);
  // last descriptor with block_begin <= blk (a prefix of the array), found
  // 64 descriptors per round trip with a ballot
  const int lane = threadIdx.x & 63;
  int lo = 0;
  for (int base = 0; base < count; base += 64) {
    const int i = base + lane;
    const bool ok = i < count && as_global(descs)[i].block_begin <= blk;
    const uint64_t mk = __ballot(ok);
    const int len = __popcll(mk);
    lo = base + len - 1;
    if (len < 64) break;
  }
  lo = __builtin_amdgcn_readfirstlane(lo);
  const sherry_gemm_desc& d = descs[lo];
  const SkProblem p{d.w, d.x, d.x_scale, d.y, d.acc, d.n, d.k, d.m, d.w_scale};
  sk_block<MT, 1>(p, blk - d.block_begin, lut, lds + kSkLutBytes);
}

}  // namespace

int skinny_blocks(int64_t n) { return static_cast<int>(ceil_div(ceil_div(n, kTileRows), kSkWaves)); }

// K splits per tile of a lone launch: the smallest power of two (up to a
// chunk's units) that gives the launch at least kSkMinBlocks workgroups, so
// that small-N products still spread over many CUs.
constexpr int64_t kSkMinBlocks = 192;

template <int MT, int S>
int launch_skinny_s(const SkProblem& p, hipStream_t s) {
  const int64_t R = ceil_div(p.n, kTileRows);
  const dim3 grid(static_cast<unsigned>(ceil_div(R, kSkWaves / S))), block(kSkThreads);
  return launch(skinny_kernel<MT, S>, grid, block, 0, s, p);
}

template <int MT>
int launch_skinny_mt(const SkProblem& p, hipStream_t s) {
  const int64_t R = ceil_div(p.n, kTileRows);
  const int64_t C = ceil_div(p.k, kTileK);
  int S = 1;
  while (S < SkCfg<MT>::UPC && S < kSkWaves && ceil_div(R, kSkWaves / S) < kSkMinBlocks &&
         C >= 2 * S)
    S *= 2;
  switch (S) {
    case 1: return launch_skinny_s<MT, 1>(p, s);
    case 2: return launch_skinny_s<MT, 2>(p, s);
    case 4: return launch_skinny_s<MT, 4>(p, s);
    default:
      if constexpr (SkCfg<MT>::UPC >= 8) return launch_skinny_s<MT, 8>(p, s);
      return launch_skinny_s<MT, 4>(p, s);
  }
}

int launch_skinny(const uint8_t* w, const int8_t* x, const float* x_scale, float w_scale,
                  float* y, int32_t* acc, int64_t m, int64_t n, int64_t k, hipStream_t s) {
  const SkProblem p{w, x, x_scale, y, acc, static_cast<int>(n), static_cast<int>(k),
                    static_cast<int>(m), w_scale};
  if (m <= 32) return launch_skinny_mt<1>(p, s);
  return launch_skinny_mt<2>(p, s);
}

int launch_skinny_batched(const sherry_gemm_desc* descs, int count, int64_t total_blocks,
                          int max_m, hipStream_t s) {
  const dim3 grid(static_cast<unsigned>(total_blocks)), block(kSkThreads);
  if (max_m <= 32) return launch(skinny_batched_kernel<1>, grid, block, 0, s, descs, count);
  return launch(skinny_batched_kernel<2>, grid, block, 0, s, descs, count);
}

}  // namespace sherry
