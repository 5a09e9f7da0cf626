// Register-decoded int8-MFMA product (Eq. 2), for any number of tokens:
// the weight stream of the decode kernel, with the multiply-accumulate on
// int8 MFMA.  Its first use is small M (5 to a few dozen tokens), where the
// weights dominate the traffic; larger M runs as a grid of token blocks (32
// tokens for products of up to 32, else 64).
//
// Work mapping.  A workgroup is W = 8 waves; wave w owns 64-row tile
// (W/S)g + w/S and part w%S of its containers along K (S = 1 unless a lone
// launch has too few tiles to fill the GPU).
// The waves walk K in lockstep chunks; the activations of a chunk (every
// staged token) arrive in LDS by DMA loads, one or three chunks ahead of
// their use.
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
typedef __attribute__((address_space(3))) void lds_void;

// Waves per workgroup (lone and grouped launches; kept apart so that each
// can be tuned on its own).
constexpr int kSkWavesLone = 8;
constexpr int kSkWavesGrouped = 8;
constexpr int kSkRing = 4;        // containers per wave in the register ring
constexpr int kSkLutBytes = 128;  // the code table, at LDS address 0
constexpr int kSkOutside = 0x7FFFFFF0;  // a buffer offset past any range: loads read zero
// Staging geometry for MT blocks of 32 tokens and W waves: a stage holds
// every staged token's KC = 1024/MT activations (32 KB), filled by LDS-DMA
// loads of 1 KB per wave instruction; NST stages form a ring, so the loads for
// chunk ch + NST - 1 are in flight while chunk ch is multiplied.
template <int MT, int NST, int W>
struct SkCfg {
  static constexpr int TOK = 32 * MT;        // staged token rows
  static constexpr int KC = 1024 / MT;       // K values per chunk (row bytes in a stage)
  static constexpr int CPR = KC / 16;        // 16-byte pieces per row
  static constexpr int UPC = KC / kTileK;    // containers per chunk
  static constexpr int STAGE = TOK * KC;
  static constexpr int SPT = STAGE / 1024 / W;  // DMA instructions per wave per chunk
  static constexpr int LDS = kSkLutBytes + NST * STAGE;
  static_assert(SPT * 1024 * W == STAGE && CPR >= 16, "stage split");
  static_assert(NST >= 2 && LDS <= 160 * 1024, "stages fit the LDS");
};

// One product of a batch (or the whole single-product launch).
struct SkProblem {
  const uint8_t* w;
  const int8_t* x;
  const float* x_scale;
  float* y;
  int32_t* acc;
  int n, k, m;
  WScale ws;
  const float* gs;  // per-group scales [n][ceil(k/128)] (grouped kernels only)
};

// Waits until at most N vector-memory loads of this wave are outstanding
// (loads complete in issue order); the other counters are left alone.
template <int N>
__device__ __forceinline__ void sk_wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  // simm16: vmcnt[3:0] at bits 3:0, expcnt 6:4, lgkmcnt 11:8, vmcnt[5:4] at 15:14
  constexpr int kImm = (N & 15) | (7 << 4) | (15 << 8) | (((N >> 4) & 3) << 14);
  __builtin_amdgcn_s_waitcnt(static_cast<int16_t>(kImm));
}

// One 16-byte LDS-DMA load per lane: lane i's bytes land at dst + 16 i.
__device__ __forceinline__ void sk_dma(__amdgpu_buffer_rsrc_t r, int8_t* dst, int voffset) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void*)dst, 16, voffset, 0, 0, 0);
}

template <int j0, int... js>
__device__ __forceinline__ void sk_offsets(const uint32_t (&d)[5], uint32_t* a4,
                                           std::integer_sequence<int, js...>) {
  ((a4[js] = code_x4<j0 + js>(d)), ...);
}

// Table lookups of container d's 32 codes (lane i = row i): wv[j] holds the
// int8x4 weights of K values 4j .. 4j+3 of the lane's row.
__device__ __forceinline__ void sk_lookup(const uint32_t (&d)[5], const uint32_t* lut,
                                          uint32_t (&wv)[32]) {
  uint32_t a4[32];
  sk_offsets<0>(d, a4, std::make_integer_sequence<int, 32>{});
#pragma unroll
  for (int j = 0; j < 32; ++j)
    wv[j] = *reinterpret_cast<const uint32_t*>(reinterpret_cast<const char*>(lut) + a4[j]);
}

template <int j0, int... is>
__device__ __forceinline__ void sk_lookup8(const uint32_t (&d)[5], const uint32_t* lut,
                                           uint32_t (&wv)[32], std::integer_sequence<int, is...>) {
  ((wv[j0 + is] = *reinterpret_cast<const uint32_t*>(reinterpret_cast<const char*>(lut) +
                                                     code_x4<j0 + is>(d))),
   ...);
}

// Step s (K values 32s .. 32s+31) of one container: words 8s..8s+3 of wv hold
// K 32s..32s+15 of this lane's row, 8s+4..8s+7 the next 16; after the swap
// the first four hold rows 0-31 and the last four rows 32-63, in the operand
// layout.  Once the step's MFMAs are issued the 8 words take the next
// container's lookups; the compiler schedules the lookups among the
// following steps (no scheduling barrier here: measured 2-5% faster, with
// the same order of global loads and waits).
template <int MT, int s>
__device__ __forceinline__ void sk_mfma_step(uint32_t (&wv)[32], const uint32_t (&dn)[5],
                                             const uint32_t* lut, const v4i (&xv)[MT],
                                             v16i (&c)[2][MT]) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const auto r =
        __builtin_amdgcn_permlane32_swap(wv[8 * s + i], wv[8 * s + 4 + i], false, false);
    wv[8 * s + i] = r[0];
    wv[8 * s + 4 + i] = r[1];
  }
  const v4i wl = {static_cast<int>(wv[8 * s]), static_cast<int>(wv[8 * s + 1]),
                  static_cast<int>(wv[8 * s + 2]), static_cast<int>(wv[8 * s + 3])};
  const v4i wh = {static_cast<int>(wv[8 * s + 4]), static_cast<int>(wv[8 * s + 5]),
                  static_cast<int>(wv[8 * s + 6]), static_cast<int>(wv[8 * s + 7])};
#pragma unroll
  for (int tb = 0; tb < MT; ++tb) {
    c[0][tb] = __builtin_amdgcn_mfma_i32_32x32x32_i8(xv[tb], wl, c[0][tb], 0, 0, 0);
    c[1][tb] = __builtin_amdgcn_mfma_i32_32x32x32_i8(xv[tb], wh, c[1][tb], 0, 0, 0);
  }
  sk_lookup8<8 * s>(dn, lut, wv, std::make_integer_sequence<int, 8>{});
}

// Accumulates one container's 128 K values (looked-up weights wv) against the
// staged activations into c[row group][token block], looking up the next
// container's codes dn into wv on the way.  All of the container's activation
// fragments are read first (lane l: token row 32tb + l%32 at row base xrow,
// the 16-byte piece for step s at xrow + lo[s], the stage's swizzle resolved
// per lane), so only the first step waits for the LDS.
template <int MT, int NST>
__device__ __forceinline__ void sk_mfma(uint32_t (&wv)[32], const uint32_t (&dn)[5],
                                        const uint32_t* lut, const int8_t* xrow,
                                        const int (&lo)[4], v16i (&c)[2][MT]) {
  using G = SkCfg<MT, NST, kSkWavesLone>;  // KC only
  v4i xv[4][MT];
#pragma unroll
  for (int s = 0; s < 4; ++s)
#pragma unroll
    for (int tb = 0; tb < MT; ++tb)
      xv[s][tb] = *reinterpret_cast<const v4i*>(xrow + lo[s] + tb * 32 * G::KC);
  sk_mfma_step<MT, 0>(wv, dn, lut, xv[0], c);
  sk_mfma_step<MT, 1>(wv, dn, lut, xv[1], c);
  sk_mfma_step<MT, 2>(wv, dn, lut, xv[2], c);
  sk_mfma_step<MT, 3>(wv, dn, lut, xv[3], c);
}

// Barrier for LDS traffic only (outstanding global loads stay in flight).
__device__ __forceinline__ void sk_lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Waits for this wave's LDS reads and writes (the other counters are left
// alone).
__device__ __forceinline__ void sk_wait_lgkm() {
  __builtin_amdgcn_s_waitcnt(15 | (7 << 4) | (0 << 8) | (3 << 14));
}

// Workgroup barrier between stage chunks.  A workgroup-scope release fence
// would also wait for every DMA still in flight (they write LDS), so the
// ordering is explicit instead: the caller has waited for its own DMAs of
// the chunk about to be read (sk_wait_vm), every LDS read of the previous
// chunk has returned (its results fed MFMAs issued before this point), and
// the compiler moves no memory access across the barrier.
__device__ __forceinline__ void sk_stage_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_sched_barrier(0);
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_sched_barrier(0);
  asm volatile("" ::: "memory");
}

// Workgroup g of problem p: tiles T*g .. T*g+T-1 (T = 8/S), each split along
// K over S waves (wave w: tile w/S, split w%S).  Split s owns units
// [s*U, min((s+1)*U, C)) with U = ceil(C/S); all waves walk their ranges in
// lockstep chunks of UPS = UPC/S units, and a stage holds, for every token,
// the S splits' windows side by side.  With S > 1 the partial accumulators
// meet in LDS (over the stages) and split 0 writes the tile.
//
// Stage layout: token row t at t*KC; its 16-byte piece c (K window offset
// 16c) at piece c ^ (t & 15), so that the 16 lanes of a read phase (16
// consecutive tokens, one piece each) hit 16 different bank groups.
//
// Load order per container step: two weight loads (the ring), then this
// step's share of the DMA for the chunk NST - 1 ahead.  Both are issued
// unconditionally (weight units past the split's end come through an empty
// resource and read zeros; DMA pieces past k read zeros or unused rows), so the
// number of loads issued after the last DMA of any chunk is fixed and the
// wait before that chunk's barrier is a constant vmcnt.
//
// With GR the weights carry per-group scales p.gs (one per row and 128
// weights, i.e. per unit): after each unit's MFMAs the int32 accumulators
// are scaled into fp32 ones (unit order) and cleared; two scale loads per
// unit ride with the weight loads.  (The int32 totals, when asked for, come
// from a second, unscaled launch.)
template <int MT, int S, int NST, int W, bool GR = false>
__device__ __forceinline__ void sk_block(const SkProblem& p, int g, const uint32_t* lut,
                                         int8_t* xs) {
  using G = SkCfg<MT, NST, W>;
  static_assert(S >= 1 && G::UPC % S == 0, "splits divide a chunk");
  constexpr int T = W / S;           // tiles per workgroup
  constexpr int UPS = G::UPC / S;    // units per split per chunk
  constexpr int WIN = UPS * kTileK;  // K values per split window
  constexpr int D = NST - 1;         // chunks between a DMA and its use
  // DMA instructions at each container position of a chunk
  constexpr int PER = UPS >= G::SPT ? 1 : G::SPT / UPS;
  constexpr int PL = UPS >= G::SPT ? G::SPT - 1 : UPS - 1;  // position of the last
  // loads issued after chunk ch's last DMA when chunk ch is reached: steady
  // state, and chunks 1..D-1 (whose DMAs the prologue issued)
  constexpr int LPC = GR ? 4 : 2;  // vector loads per unit besides the DMA
  constexpr int NSTEADY = LPC * (UPS - 1 - PL) + (D - 1) * (LPC * UPS + G::SPT);
  constexpr int NPRO = (D - 1) * G::SPT + LPC * kSkRing;
  static_assert(G::SPT % PER == 0 && PER * (PL + 1) == G::SPT, "DMA spread");
  // vmcnt holds at most 63: waiting for fewer outstanding loads than the
  // count is always safe (the loads complete in order), only stricter
  constexpr int NSTEADY_W = NSTEADY < 63 ? NSTEADY : 63;
  constexpr int NPRO_W = NPRO < 63 ? NPRO : 63;
  static_assert(!GR || MT == 1, "per-group scales use 32-token blocks");

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int C = (p.k + kTileK - 1) / kTileK;
  const int R = (p.n + kTileRows - 1) / kTileRows;
  const int U = (C + S - 1) / S;     // units per split
  const int r = g * T + wave / S;
  const int sp = wave % S;
  const int u0 = sp * U, u1 = (u0 + U < C) ? u0 + U : C;
  // the scales of this lane's epilogue stores (tokens (lane >> 3) + 8i of
  // each 32-token block, rows 32h + 4(lane & 7) + u of the tile), loaded
  // before any other load: one counter tracks a wave's loads and stores, so a
  // load issued between the stores would wait for every store before it
  float sxl[MT][4], swl[2][4];
#pragma unroll
  for (int tb = 0; tb < MT; ++tb)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int tok = 32 * tb + (lane >> 3) + 8 * i;
      sxl[tb][i] = tok < p.m ? as_global(p.x_scale)[tok] : 0.0f;
    }
#pragma unroll
  for (int h = 0; h < 2; ++h)
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int row = r * kTileRows + 32 * h + 4 * (lane & 7) + u;
      swl[h][u] = (!GR && row < p.n) ? p.ws.at(row) : 0.0f;
    }
  const bool live = r < R && u0 < u1;
  const UnitRun rs{p.w + (int64_t(r < R ? r : 0) * C + (live ? u0 : 0)) * kUnitBytes,
                   live ? u1 - u0 : 0};
  const int nch = (U + UPS - 1) / UPS;
  // the activations of the staged tokens; rows past m read zeros
  const __amdgpu_buffer_rsrc_t rx = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<int8_t*>(p.x), 0, p.m * p.k, kBufferWord3);

  // DMA instruction i of this wave fills 1 KB block i*8 + wave of a stage:
  // lane slot q = 64 * block + lane is token q / CPR, swizzled piece q % CPR,
  // i.e. window ws = o / WIN at offset wo = o % WIN.  Its K offset at chunk ch
  // is kb + ch*WIN with kb = ws*U*128 + wo; pieces past the end of their
  // split's range or past k are loaded from an offset outside the buffer,
  // so they arrive as zeros (lim = K values left in the lane's window).
  int dvo[G::SPT], lim[G::SPT];
#pragma unroll
  for (int i = 0; i < G::SPT; ++i) {
    const int q = 64 * (i * W + wave) + lane;
    const int t = q / G::CPR;
    const int o = 16 * ((q % G::CPR) ^ (t & 15));
    const int ws = o / WIN;
    const int kb = ws * U * kTileK + o % WIN;
    const int kend = ((ws + 1) * U < C ? (ws + 1) * U * kTileK : p.k);
    dvo[i] = t * p.k + kb;
    lim[i] = (kend < p.k ? kend : p.k) - kb;
  }
  int8_t* const xw = xs + 1024 * wave;  // + stage + 8 KB per instruction
  auto dma = [&](int ch, int i, int voff, int left) {
    sk_dma(rx, xw + (ch % NST) * G::STAGE + i * 1024 * W,
           ch * WIN < left ? voff + ch * WIN : kSkOutside);
  };

  // reader: token row lane%32 (plus 32tb), piece (8b + 2s + lane/32) ^ (lane & 15)
  // for window piece base 8b
  const int sw = lane & 15;
  int lo[4];
#pragma unroll
  for (int s = 0; s < 4; ++s) lo[s] = 16 * ((2 * s + (lane >> 5)) ^ (sw & 7));
  const int8_t* xlane = xs + (lane & 31) * G::KC;

  // A row length k that is not a multiple of 16 leaves, in the 16-byte piece
  // that holds K = k, bytes of the next token's row: they are cleared in the
  // stage once that piece has landed (chunk chl).
  const int kr = p.k & 15;
  const int sl = (C - 1) / U, jl = (C - 1) - sl * U;
  const int chl = kr ? jl / UPS : -1;
  auto clear_tail = [&]() {
    const int o = sl * WIN + (jl % UPS) * kTileK + ((p.k & ~15) - (C - 1) * kTileK);
    const int nd = (16 - kr) / 4;  // dwords to clear per token row
    int8_t* st = xs + (chl % NST) * G::STAGE;
    for (int e = tid; e < G::TOK * nd; e += 64 * W) {
      const int t = e / nd, b = kr + 4 * (e % nd);
      *reinterpret_cast<uint32_t*>(st + t * G::KC + 16 * ((o / 16) ^ (t & 15)) + b) = 0;
    }
    sk_wait_lgkm();
    sk_stage_barrier();
  };

  v16i c[2][MT];
#pragma unroll
  for (int h = 0; h < 2; ++h)
#pragma unroll
    for (int tb = 0; tb < MT; ++tb) c[h][tb] = v16i{};
  // per-group: fp32 sums, and the scales of the ring's units for rows
  // 32h + lane%32 (a resource over the tile's scale rows; rows past n read
  // zero)
  typedef float v16f __attribute__((ext_vector_type(16)));
  v16f cf[2][GR ? MT : 1];
  float gsr[kSkRing][2];
  __amdgpu_buffer_rsrc_t grs;
  if constexpr (GR) {
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int tb = 0; tb < MT; ++tb) cf[h][tb] = v16f{};
    const int rows = (r < R) ? p.n - r * kTileRows : 0;
    grs = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<float*>(p.gs) + int64_t(r < R ? r : 0) * kTileRows * C, 0,
        (rows < kTileRows ? rows : kTileRows) * C * 4, kBufferWord3);
  }
  auto load_scales = [&](float (&gq)[2], int unit) {
#pragma unroll
    for (int h = 0; h < 2; ++h)
      gq[h] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                                            grs, 4 * ((32 * h + (lane & 31)) * C + u0 + unit),
                                            0, 0));
  };

#pragma unroll
  for (int ch = 0; ch < D; ++ch)
#pragma unroll
    for (int i = 0; i < G::SPT; ++i) dma(ch, i, dvo[i], lim[i]);
  __builtin_amdgcn_sched_barrier(0);
  uint32_t ring[kSkRing][5];
#pragma unroll
  for (int u = 0; u < kSkRing; ++u) {
    load_unit(ring[u], rs, u, lane);
    if constexpr (GR) load_scales(gsr[u], u);
    __builtin_amdgcn_sched_barrier(0);
  }
  sk_wait_vm<NPRO_W>();
  sk_wait_lgkm();
  sk_stage_barrier();  // chunk 0 and the table are ready
  if (chl == 0) clear_tail();

  // Software pipeline: step jj multiplies container jj (weights looked up in
  // the previous step) and looks up container jj + 1, so the table reads and
  // field extraction overlap the MFMAs.  Units past the split's end multiply
  // zero activations; waves past the last tile compute values never stored.
  uint32_t wv[32];
  sk_lookup(ring[0], lut, wv);
  const int nunits = nch * UPS;  // unit j of the split lives in chunk j / UPS
  for (int j = 0; j < nunits; j += kSkRing) {
#pragma unroll
    for (int u = 0; u < kSkRing; ++u) {
      const int jj = j + u;
      const int ch = jj / UPS, pos = jj % UPS;
      if (pos == 0 && jj > 0) {
        if (ch >= D) {
          sk_wait_vm<NSTEADY_W>();
        } else {
          // chunk ch < D: its DMA went out in the prologue
          if constexpr (D > 1) {
            if (ch == 1) sk_wait_vm<NPRO + LPC * UPS < 64 ? NPRO + LPC * UPS : 63>();
            if constexpr (D > 2)
              if (ch == 2)
                sk_wait_vm<NPRO + 2 * LPC * UPS < 64 ? NPRO + 2 * LPC * UPS : 63>();
          }
        }
        sk_stage_barrier();
        if (ch == chl) clear_tail();
      }
      __builtin_amdgcn_sched_barrier(0);
      load_unit(ring[u], rs, jj + kSkRing, lane);  // container jj's codes are used
      __builtin_amdgcn_sched_barrier(0);
      const int wb = sp * WIN / 16 + 8 * pos;  // window piece base (multiple of 8)
      const int8_t* xrow = xlane + (ch % NST) * G::STAGE + 128 * ((wb >> 3) ^ (sw >> 3));
      sk_mfma<MT, NST>(wv, ring[(u + 1) % kSkRing], lut, xrow, lo, c);
      __builtin_amdgcn_sched_barrier(0);
      if constexpr (GR) {
#pragma unroll
        for (int h = 0; h < 2; ++h)
#pragma unroll
          for (int tb = 0; tb < MT; ++tb) {
#pragma unroll
            for (int e = 0; e < 16; ++e)
              cf[h][tb][e] = __builtin_fmaf(static_cast<float>(c[h][tb][e]), gsr[u][h],
                                            cf[h][tb][e]);
            c[h][tb] = v16i{};
          }
        load_scales(gsr[u], jj + kSkRing);
        __builtin_amdgcn_sched_barrier(0);
      }
      if (pos <= PL) {
#pragma unroll
        for (int i = 0; i < PER; ++i) {
          const int id = pos * PER + i;
          dma(ch + D, id, dvo[id], lim[id]);
        }
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  sk_wait_vm<0>();  // no DMA may land in the LDS after this point

  if constexpr (S > 1 && GR) {
    // fp32 partial sums of the S splits, in split order
    float* redf = reinterpret_cast<float*>(xs);
    sk_lds_barrier();
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int e = 0; e < 16; ++e) redf[((wave * 2 + h) * 16 + e) * 64 + lane] = cf[h][0][e];
    sk_lds_barrier();
    if (sp == 0) {
#pragma unroll
      for (int q = 1; q < S; ++q)
#pragma unroll
        for (int h = 0; h < 2; ++h)
#pragma unroll
          for (int e = 0; e < 16; ++e)
            cf[h][0][e] += redf[(((wave + q) * 2 + h) * 16 + e) * 64 + lane];
    }
  }
  if constexpr (S > 1 && !GR) {
    // partial sums of the S splits of a tile through LDS (the stages are
    // free now), one token block at a time: [wave][h][element][lane]
    int32_t* red = reinterpret_cast<int32_t*>(xs);
    static_assert(W * 2 * 16 * 64 * 4 <= NST * G::STAGE, "reduction fits the stages");
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
  // e = accumulator element.  Each 32-token x 32-row block is staged in the
  // wave's own LDS region (row stride 40 words: the half-waves' tokens, 4
  // apart, use disjoint banks) and read back as 16-byte pieces of 4 rows, so
  // that every lane stores 16 bytes and 8 lanes write 128 contiguous bytes;
  // a wave's LDS accesses run in order, so the region needs no barrier of
  // its own.
  sk_lds_barrier();  // every wave is done with the stages and the reduction
  if (r >= R || sp != 0) return;
  constexpr int SW = 40;
  static_assert((W / S) * 32 * SW * 4 <= NST * G::STAGE, "epilogue regions fit the stages");
  int32_t* strip = reinterpret_cast<int32_t*>(xs) + (wave / S) * 32 * SW;
  const bool vec = (p.n % 4 == 0) && (reinterpret_cast<uintptr_t>(p.y) % 16 == 0) &&
                   (GR || !p.acc || reinterpret_cast<uintptr_t>(p.acc) % 16 == 0);
#pragma unroll
  for (int tb = 0; tb < MT; ++tb) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int tl = 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
        if constexpr (GR) {
          // copy the element out first: a bit cast of a vector element in
          // place reads element 0
          const float f = cf[h][0][e];
          strip[tl * SW + (lane & 31)] = __float_as_int(f);
        } else {
          strip[tl * SW + (lane & 31)] = c[h][tb][e];
        }
      }
      __asm__ volatile("" ::: "memory");
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int q = lane + 64 * i;
        const int tl = q >> 3, c4 = q & 7;
        const v4i v = *reinterpret_cast<const v4i*>(strip + tl * SW + 4 * c4);
        const int tok = 32 * tb + tl;
        const int row = r * kTileRows + 32 * h + 4 * c4;
        if (tok >= p.m || row >= p.n) continue;
        const float sx = sxl[tb][i];
        const int32_t vv[4] = {v.x, v.y, v.z, v.w};
        float o[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          if constexpr (GR) o[u] = __int_as_float(vv[u]) * sx;
          else o[u] = static_cast<float>(vv[u]) * (sx * swl[h][u]);
        }
        float* yrow = as_global_mut(p.y) + int64_t(tok) * p.n + row;
        if (vec) {
          *reinterpret_cast<float4*>(yrow) = make_float4(o[0], o[1], o[2], o[3]);
          if constexpr (!GR)
            if (p.acc) *reinterpret_cast<v4i*>(as_global_mut(p.acc) + int64_t(tok) * p.n + row) = v;
        } else {
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            if (row + u >= p.n) break;
            yrow[u] = o[u];
            if constexpr (!GR)
              if (p.acc) as_global_mut(p.acc)[int64_t(tok) * p.n + row + u] = vv[u];
          }
        }
      }
      __asm__ volatile("" ::: "memory");  // the next block overwrites these reads
    }
  }
}

// Stage ring depth: two stages (one chunk ahead) for lone 32-token launches,
// four otherwise (measured).
template <int MT, bool kGrouped>
constexpr int kSkStages = (MT == 1 && !kGrouped) ? 2 : 4;

// grid: x = groups of W/S tiles, y = blocks of 32*MT tokens
template <int MT, int S, bool GR = false>
__global__ __launch_bounds__(64 * kSkWavesLone) void skinny_kernel(SkProblem p) {
  constexpr int W = kSkWavesLone;
  constexpr int NST = kSkStages<MT, false>;
  using G = SkCfg<MT, NST, W>;
  __shared__ __attribute__((aligned(16))) int8_t lds[G::LDS];
  uint32_t* lut = reinterpret_cast<uint32_t*>(lds);
  if (threadIdx.x < 32) lut[threadIdx.x] = decode_word(threadIdx.x);
  const int t0 = blockIdx.y * G::TOK;
  p.x += int64_t(t0) * p.k;
  p.x_scale += t0;
  p.y += int64_t(t0) * p.n;
  if (p.acc) p.acc += int64_t(t0) * p.n;
  p.m = (p.m - t0 < G::TOK) ? p.m - t0 : G::TOK;
  sk_block<MT, S, NST, W, GR>(p, blockIdx.x, lut, lds + kSkLutBytes);
}

template <int MT>
__global__ __launch_bounds__(64 * kSkWavesGrouped) void skinny_batched_kernel(
    const sherry_gemm_desc* __restrict__ descs, int count) {
  constexpr int W = kSkWavesGrouped;
  constexpr int NST = kSkStages<MT, true>;
  __shared__ __attribute__((aligned(16))) int8_t lds[SkCfg<MT, NST, W>::LDS];
  uint32_t* lut = reinterpret_cast<uint32_t*>(lds);
  if (threadIdx.x < 32) lut[threadIdx.x] = decode_word(threadIdx.x);
  const int32_t blk = static_cast<int32_t>(blockIdx.x);
  // the descriptor whose block range holds blk
  const int lo = find_block_desc(descs, count, blk);
  if (lo < 0) return;
  const sherry_gemm_desc& d = descs[lo];
  // a product's blocks: its tile groups for token block 0, then for token
  // block 1, ... (blocks in flight together share their activations)
  constexpr int TOK = SkCfg<MT, NST, W>::TOK;
  const int lb = blk - d.block_begin;
  if constexpr (MT == 1) {
    // per-group scales (prepare reports a 32-token launch for them): K split
    // in two, fp32 sums per group, no int32 totals
    if (d.w_group_scales) {
      const int gg = static_cast<int>(ceil_div(ceil_div(d.n, kTileRows), W / 2));
      const int tg = lb / gg;
      const int tg0 = tg * TOK;
      const SkProblem pg{d.w,
                         d.x + int64_t(tg0) * d.k,
                         d.x_scale + tg0,
                         d.y + int64_t(tg0) * d.n,
                         nullptr,
                         d.n,
                         d.k,
                         (d.m - tg0 < TOK) ? d.m - tg0 : TOK,
                         WScale{nullptr, 0.0f},
                         d.w_group_scales};
      sk_block<1, 2, NST, W, true>(pg, lb - tg * gg, lut, lds + kSkLutBytes);
      return;
    }
  }
  const int gb = static_cast<int>(ceil_div(ceil_div(d.n, kTileRows), W));
  const int tb = lb / gb;
  const int t0 = tb * TOK;
  const SkProblem p{d.w,
                    d.x + int64_t(t0) * d.k,
                    d.x_scale + t0,
                    d.y + int64_t(t0) * d.n,
                    d.acc ? d.acc + int64_t(t0) * d.n : nullptr,
                    d.n,
                    d.k,
                    (d.m - t0 < TOK) ? d.m - t0 : TOK,
                    WScale{d.w_scales, d.w_scale},
                    nullptr};
  sk_block<MT, 1, NST, W>(p, lb - tb * gb, lut, lds + kSkLutBytes);
}

}  // namespace

// Workgroups of one product's token block in a grouped launch (products
// with per-group scales split each tile's K in two, so a workgroup holds
// half as many tiles), and the token block of a grouped launch whose
// largest product has max_m tokens.
int skinny_blocks(int64_t n, bool group_scales) {
  return static_cast<int>(
      ceil_div(ceil_div(n, kTileRows), group_scales ? kSkWavesGrouped / 2 : kSkWavesGrouped));
}
int skinny_batched_tokens(int max_m) {
  return max_m <= 32 ? SkCfg<1, kSkStages<1, true>, kSkWavesGrouped>::TOK
                     : SkCfg<2, kSkStages<2, true>, kSkWavesGrouped>::TOK;
}

// K splits per tile of a lone launch: the smallest power of two (up to a
// chunk's units) that gives the launch at least kSkMinBlocks workgroups, so
// that small-N products still spread over many CUs.
constexpr int64_t kSkMinBlocks = 192;

// Token blocks beyond the grid's y limit go to further launches.
constexpr int64_t kSkMaxGridY = 32768;

template <int MT, int S, bool GR>
int launch_skinny_s(const SkProblem& p, hipStream_t s) {
  const int64_t R = ceil_div(p.n, kTileRows);
  const int64_t TB = ceil_div(p.m, SkCfg<MT, kSkStages<MT, false>, kSkWavesLone>::TOK);
  for (int64_t b0 = 0; b0 < TB; b0 += kSkMaxGridY) {
    const int64_t nb = TB - b0 < kSkMaxGridY ? TB - b0 : kSkMaxGridY;
    const int64_t t0 = b0 * SkCfg<MT, kSkStages<MT, false>, kSkWavesLone>::TOK;
    SkProblem q = p;
    q.x += t0 * p.k;
    q.x_scale += t0;
    q.y += t0 * p.n;
    if (q.acc) q.acc += t0 * p.n;
    q.m = static_cast<int>(p.m - t0);
    const dim3 grid(static_cast<unsigned>(ceil_div(R, kSkWavesLone / S)),
                    static_cast<unsigned>(nb));
    const int rc = launch(skinny_kernel<MT, S, GR>, grid, dim3(64 * kSkWavesLone), 0, s, q);
    if (rc != SHERRY_OK) return rc;
  }
  return SHERRY_OK;
}

template <int MT, bool GR = false>
int launch_skinny_mt(const SkProblem& p, hipStream_t s) {
  const int64_t R = ceil_div(p.n, kTileRows);
  const int64_t C = ceil_div(p.k, kTileK);
  const int64_t TB = ceil_div(p.m, SkCfg<MT, kSkStages<MT, false>, kSkWavesLone>::TOK);
  // the per-group kernel always splits K at least in two (fewer units per
  // wave keep its registers in bounds)
  int S = GR ? 2 : 1;
  while (S < SkCfg<MT, kSkStages<MT, false>, kSkWavesLone>::UPC && S < kSkWavesLone &&
         ceil_div(R, kSkWavesLone / S) * TB < kSkMinBlocks &&
         C >= 2 * S)
    S *= 2;
  switch (S) {
    case 1:
      if constexpr (!GR) return launch_skinny_s<MT, 1, GR>(p, s);
      return launch_skinny_s<MT, 2, GR>(p, s);
    case 2: return launch_skinny_s<MT, 2, GR>(p, s);
    case 4:
      if constexpr (SkCfg<MT, kSkStages<MT, false>, kSkWavesLone>::UPC >= 4) return launch_skinny_s<MT, 4, GR>(p, s);
      return launch_skinny_s<MT, 2, GR>(p, s);
    default:
      if constexpr (SkCfg<MT, kSkStages<MT, false>, kSkWavesLone>::UPC >= 8) return launch_skinny_s<MT, 8, GR>(p, s);
      return launch_skinny_s<MT, 2, GR>(p, s);
  }
}

int launch_skinny(const uint8_t* w, const int8_t* x, const float* x_scale, WScale ws,
                  float* y, int32_t* acc, int64_t m, int64_t n, int64_t k, hipStream_t s) {
  const SkProblem p{w, x, x_scale, y, acc, static_cast<int>(n), static_cast<int>(k),
                    static_cast<int>(m), ws, nullptr};
  if (m <= 32) return launch_skinny_mt<1>(p, s);
  return launch_skinny_mt<2>(p, s);
}

// Per-group scales: 32-token blocks for every M (the fp32 sums and int32
// totals double the accumulator registers).
int launch_skinny_group(const uint8_t* w, const int8_t* x, const float* x_scale, const float* gs,
                        float* y, int32_t* acc, int64_t m, int64_t n, int64_t k, hipStream_t s) {
  if (acc) {
    // int32 totals from an unscaled launch (its y is overwritten below)
    const int rc = launch_skinny(w, x, x_scale, WScale{nullptr, 1.0f}, y, acc, m, n, k, s);
    if (rc != SHERRY_OK) return rc;
  }
  const SkProblem p{w, x, x_scale, y, nullptr, static_cast<int>(n), static_cast<int>(k),
                    static_cast<int>(m), WScale{nullptr, 0.0f}, gs};
  return launch_skinny_mt<1, true>(p, s);
}

int launch_skinny_batched(const sherry_gemm_desc* descs, int count, int64_t total_blocks,
                          int max_m, hipStream_t s) {
  const dim3 grid(static_cast<unsigned>(total_blocks)), block(64 * kSkWavesGrouped);
  if (max_m <= 32) return launch(skinny_batched_kernel<1>, grid, block, 0, s, descs, count);
  return launch(skinny_batched_kernel<2>, grid, block, 0, s, descs, count);
}

}  // namespace sherry
