// Prefill-path product (Eq. 2 at large M): the packed T tile is decoded once
// per workgroup into an int8 tile in LDS and multiplied with int8 MFMA.
//
// Per K-step of 128 (one unit column of the packed layout):
//  - X tile  BM x 128 int8: 16-byte buffer loads, written to LDS as is;
//  - T tile  BN x 128: BN/64 units of 1280 bytes; the PARTS threads of a T
//    row each decode 32/PARTS of its codes through the 32-entry table and
//    write int8x4 words to LDS;
//  - the waves, each owning a (BM/WGM) x (BN/WGN) block of C made of 32x32
//    fragments, run v_mfma_i32_32x32x32_i8 over four 32-wide k slices.
// LDS holds two stages of [X tile | T tile]: while the MFMAs of step s read
// one stage, the registers loaded during step s-1 are written into the other
// and the loads of step s+2 are issued, so there is one barrier per step and
// every global load has a whole step to land.  Eight waves (two per SIMD)
// let one wave's decode and LDS traffic overlap the other's MFMAs.
// LDS rows are 128 bytes, with 16-byte chunks swizzled per row (swz) so
// that fragment reads and tile writes are free of bank conflicts.
#include "sherry_internal.h"

namespace sherry {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));

constexpr int kBK = 128;
constexpr int kLutBytes = 128;

template <int BM_, int BN_, int WGM_, int WGN_, int THREADS_>
struct GemmCfg {
  static constexpr int BM = BM_, BN = BN_, WGM = WGM_, WGN = WGN_, THREADS = THREADS_;
  static_assert(WGM * WGN * 64 == THREADS, "one wave per C block");
  static constexpr int WM = BM / WGM, WN = BN / WGN;
  static_assert(WM % 32 == 0 && WN % 32 == 0, "32x32 fragments");
  static constexpr int FM = WM / 32, FN = WN / 32;
  static constexpr int XPT = BM * 8 / THREADS;  // 16-byte X chunks per thread
  static_assert(XPT >= 1 && BM * 8 % THREADS == 0, "X tile split");
  // threads per T row; each decodes CPP consecutive codes of the row.  BN is
  // a multiple of 64, so a wave's threads share one part (uniform branch)
  static constexpr int PARTS = THREADS / BN;
  static_assert(BN % 64 == 0 && THREADS % BN == 0 && (PARTS == 1 || PARTS == 2 || PARTS == 4),
                "T tile split");
  static constexpr int CPP = 32 / PARTS;
  static constexpr int LDS_X = BM * kBK, LDS_W = BN * kBK, STAGE = LDS_X + LDS_W;
};

// 16-byte chunk c of LDS row r is stored at chunk c ^ (r & 7) ^ ((r >> 3) & 1):
// a 16-byte access by 16 consecutive rows at one logical chunk then covers
// all 64 LDS banks once (rows 8 apart differ in the low chunk bit and rows
// of equal swizzle differ in parity), and 8 consecutive rows cover 32 banks.
__device__ __forceinline__ int swz(int row, int chunk) {
  return row * kBK + ((chunk ^ (row & 7) ^ ((row >> 3) & 1)) << 4);
}

// Decodes codes [j0, j0 + n) (n a multiple of 4) of the row stream in d and
// writes them as int8 to the T tile row: 16-byte chunk per 4 codes.
template <int j0, int n>
__device__ __forceinline__ void decode_codes(const uint32_t (&d)[5], const uint32_t* lut,
                                             int8_t* ws, int wrow) {
  if constexpr (n > 0) {
    uint32_t q[4];
    q[0] = *reinterpret_cast<const uint32_t*>(reinterpret_cast<const char*>(lut) + code_x4<j0>(d));
    q[1] = *reinterpret_cast<const uint32_t*>(reinterpret_cast<const char*>(lut) +
                                              code_x4<j0 + 1>(d));
    q[2] = *reinterpret_cast<const uint32_t*>(reinterpret_cast<const char*>(lut) +
                                              code_x4<j0 + 2>(d));
    q[3] = *reinterpret_cast<const uint32_t*>(reinterpret_cast<const char*>(lut) +
                                              code_x4<j0 + 3>(d));
    *reinterpret_cast<uint4*>(ws + swz(wrow, j0 >> 2)) = make_uint4(q[0], q[1], q[2], q[3]);
    decode_codes<j0 + 4, n - 4>(d, lut, ws, wrow);
  }
}

// kFullK: K % 128 == 0, every X chunk of a step is in its row, so all loads
// are branch-free buffer loads (rows past M and units past N read as zero).
// With GR, gs holds per-group scales ([N][C] fp32, one per row and K-step):
// after each K-step's MFMAs the int32 accumulators are scaled into fp32 sums
// (ascending K-steps) and cleared; y = x_scale * sum, acc_out the int32
// totals.
template <class G, bool kFullK, bool GR = false>
__global__ __launch_bounds__(G::THREADS) void gemm_kernel(
    const uint8_t* __restrict__ w, const int8_t* __restrict__ x,
    const float* __restrict__ x_scale, WScale ws, float* __restrict__ y,
    int32_t* __restrict__ acc_out, int64_t M, int64_t N, int64_t K, int MT, int NT,
    const float* __restrict__ gs = nullptr) {
  // LDS: the 32-entry code table at address 0 (table reads then need no base
  // in their address), then the two stages
  __shared__ __attribute__((aligned(16))) int8_t lds[kLutBytes + 2 * G::STAGE];
  uint32_t* lut = reinterpret_cast<uint32_t*>(lds);
  int8_t* smem = lds + kLutBytes;
  if (threadIdx.x < 32) lut[threadIdx.x] = decode_word(threadIdx.x);

  // tile of this block; XCD-aware: consecutive blocks land on different XCDs,
  // so give each XCD a contiguous range of tiles (same T columns, all M rows)
  const int T = MT * NT;
  const int b = blockIdx.x;
  int L = b;
  if (T % 8 == 0) L = (b & 7) * (T >> 3) + (b >> 3);
  const int mt = L % MT, nt = L / MT;
  const int64_t m0 = int64_t(mt) * G::BM, n0 = int64_t(nt) * G::BN;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wr = wave / G::WGN, wc = wave % G::WGN;

  const int64_t C = (K + kBK - 1) / kBK;           // K-steps == unit columns
  const int64_t R = (N + kTileRows - 1) / kTileRows;  // unit rows

  // T row of this thread within the tile and its part (wave-uniform)
  const int wrow = tid % G::BN;
  const int part = __builtin_amdgcn_readfirstlane(tid / G::BN);
  const int wi = wrow % kTileRows;  // row within its unit (n0 is a multiple of 64)

  // the scales of the tile's rows and columns, for the epilogue: loaded
  // first and parked in LDS with the first stage, because one counter tracks
  // a wave's loads and stores, so a load between the epilogue's stores would
  // wait for every store before it
  static_assert(G::THREADS >= G::BM && G::THREADS >= G::BN, "one scale per thread");
  __shared__ float sxs[G::BM];
  __shared__ float sws[G::BN];
  float sxp = 0.0f, swp = 0.0f;
  if (tid < G::BM && m0 + tid < M) sxp = x_scale[m0 + tid];
  if (tid < G::BN && n0 + tid < N) swp = ws.at(n0 + tid);

  uint4 xr[G::XPT];
  uint32_t wd[5];
  const bool k16 = (K % 16) == 0;

  // buffer resources spanning this tile's X rows and T unit rows
  const int64_t xrows = (M - m0 < G::BM) ? M - m0 : G::BM;
  const __amdgpu_buffer_rsrc_t xrs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<int8_t*>(x) + m0 * K, 0, static_cast<int>(xrows * K), kBufferWord3);
  const int64_t u0 = n0 / kTileRows;
  const int64_t urows = (R - u0 < G::BN / kTileRows) ? R - u0 : G::BN / kTileRows;
  const __amdgpu_buffer_rsrc_t wrs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(w) + u0 * C * kUnitBytes, 0,
      static_cast<int>(urows * C * kUnitBytes), kBufferWord3);
  const int wvo = static_cast<int>((wrow / kTileRows) * C * kUnitBytes);  // unit row in tile

  auto load_step = [&](int64_t ks) {
    const int kb = static_cast<int>(ks * kBK);
#pragma unroll
    for (int v = 0; v < G::XPT; ++v) {
      const int q = tid + G::THREADS * v;
      const int row = q >> 3, ch = q & 7;
      if constexpr (kFullK) {
        const u32x4 val = __builtin_amdgcn_raw_buffer_load_b128(
            xrs, static_cast<int>(row * K) + ch * 16, kb, 0);
        xr[v] = make_uint4(val.x, val.y, val.z, val.w);
      } else {
        const int64_t gm = m0 + row, gk = kb + ch * 16;
        uint4 val = make_uint4(0, 0, 0, 0);
        if (gm < M) {
          const int8_t* src = x + gm * K + gk;
          if (k16 && gk + 16 <= K) {
            val = *reinterpret_cast<const uint4*>(src);
          } else {
            uint32_t t4[4] = {0, 0, 0, 0};
#pragma unroll
            for (int e = 0; e < 4; ++e)
              if (gk + 4 * e < K) t4[e] = *reinterpret_cast<const uint32_t*>(src + 4 * e);
            val = make_uint4(t4[0], t4[1], t4[2], t4[3]);
          }
        }
        xr[v] = val;
      }
    }
    const u32x4 h = __builtin_amdgcn_raw_buffer_load_b128(wrs, wvo + 16 * wi, ks * kUnitBytes, 0);
    wd[0] = h.x;
    wd[1] = h.y;
    wd[2] = h.z;
    wd[3] = h.w;
    wd[4] = __builtin_amdgcn_raw_buffer_load_b32(wrs, wvo + kHeadBytes + 4 * wi,
                                                 ks * kUnitBytes, 0);
  };

  // writes the registers of one step into a stage: X as is, T decoded
  auto store_step = [&](int8_t* stage) {
    int8_t* xs = stage;
    int8_t* ws = stage + G::LDS_X;
#pragma unroll
    for (int v = 0; v < G::XPT; ++v) {
      const int q = tid + G::THREADS * v;
      *reinterpret_cast<uint4*>(xs + swz(q >> 3, q & 7)) = xr[v];
    }
    if (part == 0) {
      decode_codes<0, G::CPP>(wd, lut, ws, wrow);
    } else if constexpr (G::PARTS == 2) {
      decode_codes<16, 16>(wd, lut, ws, wrow);
    } else if constexpr (G::PARTS == 4) {
      if (part == 1) decode_codes<8, 8>(wd, lut, ws, wrow);
      else if (part == 2) decode_codes<16, 8>(wd, lut, ws, wrow);
      else decode_codes<24, 8>(wd, lut, ws, wrow);
    }
  };

  v16i acc[G::FM][G::FN];
#pragma unroll
  for (int a = 0; a < G::FM; ++a)
#pragma unroll
    for (int bb = 0; bb < G::FN; ++bb) acc[a][bb] = v16i{};

  const int frow = lane & 31, fhalf = lane >> 5;
  // MFMAs of one step from a stage: four 32-wide k slices.  The fragments of
  // slice t+1 are read into the other register set before the MFMAs of
  // slice t are issued, so the LDS latency hides behind those MFMAs.
  auto compute = [&](const int8_t* stage) {
    const int8_t* xs = stage;
    const int8_t* ws = stage + G::LDS_X;
    v4i af[2][G::FM], bf[2][G::FN];
    auto read = [&](int t, int set) {
#pragma unroll
      for (int a = 0; a < G::FM; ++a) {
        const int row = wr * G::WM + a * 32 + frow;
        af[set][a] = *reinterpret_cast<const v4i*>(xs + swz(row, 2 * t + fhalf));
      }
#pragma unroll
      for (int bb = 0; bb < G::FN; ++bb) {
        const int row = wc * G::WN + bb * 32 + frow;
        bf[set][bb] = *reinterpret_cast<const v4i*>(ws + swz(row, 2 * t + fhalf));
      }
    };
    read(0, 0);
#pragma unroll
    for (int t = 0; t < kBK / 32; ++t) {
      if (t + 1 < kBK / 32) read(t + 1, (t + 1) & 1);
#pragma unroll
      for (int a = 0; a < G::FM; ++a)
#pragma unroll
        for (int bb = 0; bb < G::FN; ++bb)
          acc[a][bb] = __builtin_amdgcn_mfma_i32_32x32x32_i8(af[t & 1][a], bf[t & 1][bb],
                                                             acc[a][bb], 0, 0, 0);
    }
    // schedule: slice 0's reads, then per slice the next slice's reads
    // interleaved with this slice's MFMAs (the scheduler would otherwise
    // reuse one register set and wait on every read)
    __builtin_amdgcn_sched_group_barrier(0x100, G::FM + G::FN, 0);
#pragma unroll
    for (int t = 0; t < kBK / 32; ++t) {
      if (t + 1 < kBK / 32) {
#pragma unroll
        for (int i = 0; i < G::FM + G::FN; ++i) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
          __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        }
        __builtin_amdgcn_sched_group_barrier(0x008, G::FM * G::FN - (G::FM + G::FN), 0);
      } else {
        __builtin_amdgcn_sched_group_barrier(0x008, G::FM * G::FN, 0);
      }
    }
  };

  // per-group: fp32 sums and int32 totals per accumulator element; lane's
  // column of fragment bb
  typedef float v16f __attribute__((ext_vector_type(16)));
  v16f cf[GR ? G::FM : 1][GR ? G::FN : 1];
  v16i tot[GR ? G::FM : 1][GR ? G::FN : 1];
  float gcur[G::FN];
  if constexpr (GR) {
#pragma unroll
    for (int a = 0; a < G::FM; ++a)
#pragma unroll
      for (int bb = 0; bb < G::FN; ++bb) {
        cf[a][bb] = v16f{};
        tot[a][bb] = v16i{};
      }
  }
  // scale of K-step kk for each fragment column (0 past N)
  auto load_scales = [&](int64_t kk) {
    if constexpr (GR) {
#pragma unroll
      for (int bb = 0; bb < G::FN; ++bb) {
        const int64_t col = n0 + wc * G::WN + bb * 32 + frow;
        gcur[bb] = col < N ? gs[col * C + kk] : 0.0f;
      }
    }
  };
  auto flush = [&]() {
    if constexpr (GR) {
#pragma unroll
      for (int a = 0; a < G::FM; ++a)
#pragma unroll
        for (int bb = 0; bb < G::FN; ++bb)
#pragma unroll
          for (int e = 0; e < 16; ++e) {
            cf[a][bb][e] = __builtin_fmaf(static_cast<float>(acc[a][bb][e]), gcur[bb],
                                          cf[a][bb][e]);
            tot[a][bb][e] += acc[a][bb][e];
            acc[a][bb][e] = 0;
          }
    }
  };

  load_step(0);
  __syncthreads();  // lut ready
  store_step(smem);
  if (tid < G::BM) sxs[tid] = sxp;
  if (tid < G::BN) sws[tid] = swp;
  if (C > 1) load_step(1);
  __syncthreads();

  // steady state: the stage of step ks + 1 is filled from registers (loaded
  // one step earlier), the loads of step ks + 2 are issued, then the MFMAs
  // of step ks run; one barrier per step
  // Half of the waves (one per SIMD) run the MFMAs first and fill the next
  // stage after them, so that on every SIMD one wave's decode and LDS writes
  // overlap the other wave's MFMAs.
  const bool mfma_first = G::THREADS >= 512 && (wave & 4);
  int64_t ks = 0;
  for (; ks + 2 < C; ++ks) {
    if (!mfma_first) {
      store_step(smem + ((ks + 1) & 1) * G::STAGE);
      // issue the loads before the MFMAs, so they have a whole step to land
      __builtin_amdgcn_sched_barrier(0);
      load_step(ks + 2);
    }
    load_scales(ks);
    __builtin_amdgcn_sched_barrier(0);
    compute(smem + (ks & 1) * G::STAGE);
    __builtin_amdgcn_sched_barrier(0);
    flush();
    if (mfma_first) {
      store_step(smem + ((ks + 1) & 1) * G::STAGE);
      __builtin_amdgcn_sched_barrier(0);
      load_step(ks + 2);
    }
    __syncthreads();
  }
  if (ks + 1 < C) {
    store_step(smem + ((ks + 1) & 1) * G::STAGE);
    load_scales(ks);
    compute(smem + (ks & 1) * G::STAGE);
    flush();
    __syncthreads();
    ++ks;
  }
  load_scales(ks);
  compute(smem + (ks & 1) * G::STAGE);
  flush();

  // ---- epilogue, staged through LDS so that every lane stores 16 bytes of
  // one row and a wave writes whole rows.  Lane holds C[i][j] of fragment
  // (a, bb) with j = lane%32 and i = 8*(r/4) + 4*(lane/32) + r%4 for
  // accumulator element r.  Each wave copies one 32-row strip of its block
  // (32 x WN int32, row stride WN + 8 words, so that the half-waves' rows, 4
  // apart, use disjoint banks) into its own LDS region and reads it back as
  // 16-byte row pieces; a wave's LDS accesses run in order, so the strip
  // needs no barrier of its own.
  __syncthreads();  // every wave is done reading the stages
  constexpr int SW = G::WN + 8;
  static_assert(G::THREADS / 64 * 32 * SW * 4 <= 2 * G::STAGE, "epilogue strips fit in LDS");
  int32_t* strip = reinterpret_cast<int32_t*>(smem) + wave * 32 * SW;
  const bool vec = (N % 4 == 0) && (reinterpret_cast<uintptr_t>(y) % 16 == 0) &&
                   (!acc_out || reinterpret_cast<uintptr_t>(acc_out) % 16 == 0);
  constexpr int RP = G::WN / 4;  // 16-byte pieces per strip row
  // pass 0 writes y (and, without per-group scales, the int32 sums); with
  // per-group scales pass 0 stages the fp32 sums and pass 1 the int32 totals
  const int passes = (GR && acc_out) ? 2 : 1;
  for (int pass = 0; pass < passes; ++pass) {
#pragma unroll
    for (int a = 0; a < G::FM; ++a) {
#pragma unroll
      for (int bb = 0; bb < G::FN; ++bb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          int32_t v;
          if constexpr (GR) {
            const float f = cf[a][bb][r];  // copied out: a vector element is not bit-cast in place
            v = pass == 0 ? __float_as_int(f) : tot[a][bb][r];
          } else {
            v = acc[a][bb][r];
          }
          strip[(8 * (r >> 2) + 4 * fhalf + (r & 3)) * SW + bb * 32 + frow] = v;
        }
      __asm__ volatile("" ::: "memory");
#pragma unroll
      for (int i = 0; i < 32 * RP / 64; ++i) {
        const int p = lane + 64 * i;
        const int row = p / RP, c4 = p % RP;
        const v4i v = *reinterpret_cast<const v4i*>(strip + row * SW + 4 * c4);
        const int64_t gm = m0 + wr * G::WM + a * 32 + row;
        const int64_t gn = n0 + wc * G::WN + 4 * c4;
        if (gm >= M || gn >= N) continue;
        const int32_t vv[4] = {v.x, v.y, v.z, v.w};
        if (GR && pass == 1) {  // int32 totals only
          if (vec) {
            *reinterpret_cast<v4i*>(acc_out + gm * N + gn) = v;
          } else {
#pragma unroll
            for (int e = 0; e < 4; ++e)
              if (gn + e < N) acc_out[gm * N + gn + e] = vv[e];
          }
          continue;
        }
        const float sx = sxs[wr * G::WM + a * 32 + row];
        float o[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          if constexpr (GR) o[e] = __int_as_float(vv[e]) * sx;
          else o[e] = static_cast<float>(vv[e]) * (sx * sws[wc * G::WN + 4 * c4 + e]);
        }
        if (vec) {
          *reinterpret_cast<float4*>(y + gm * N + gn) = make_float4(o[0], o[1], o[2], o[3]);
          if (!GR && acc_out) *reinterpret_cast<v4i*>(acc_out + gm * N + gn) = v;
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            if (gn + e >= N) break;
            y[gm * N + gn + e] = o[e];
            if (!GR && acc_out) acc_out[gm * N + gn + e] = vv[e];
          }
        }
      }
      __asm__ volatile("" ::: "memory");  // the next strip overwrites these reads
    }
  }
}

template <class G>
int launch_cfg(const uint8_t* w, const int8_t* x, const float* x_scale, WScale ws,
               float* y, int32_t* acc, int64_t m, int64_t n, int64_t k, hipStream_t s) {
  const int MT = static_cast<int>(ceil_div(m, G::BM));
  const int NT = static_cast<int>(ceil_div(n, G::BN));
  const dim3 grid(static_cast<unsigned>(MT) * NT), block(G::THREADS);
  if (k % kBK == 0)
    return launch(gemm_kernel<G, true>, grid, block, 0, s, w, x, x_scale, ws, y, acc, m, n,
                  k, MT, NT, static_cast<const float*>(nullptr));
  return launch(gemm_kernel<G, false>, grid, block, 0, s, w, x, x_scale, ws, y, acc, m, n, k,
                MT, NT, static_cast<const float*>(nullptr));
}

using CfgLarge = GemmCfg<256, 256, 2, 4, 512>;  // wave block 128 x 64
using CfgMid = GemmCfg<128, 256, 2, 4, 512>;    // wave block 64 x 64
using CfgSmall = GemmCfg<128, 128, 2, 4, 512>;  // wave block 64 x 32
using CfgSkinny = GemmCfg<32, 256, 1, 4, 256>;  // wave block 32 x 64

constexpr int64_t kCUs = 256;

// Rounds of one-workgroup-per-CU waves a configuration needs, weighted by
// its tile area (a proxy for time when every configuration keeps its MFMAs
// similarly busy).
template <class G>
int64_t gemm_cost(int64_t m, int64_t n) {
  return ceil_div(ceil_div(m, G::BM) * ceil_div(n, G::BN), kCUs) * G::BM * G::BN;
}

}  // namespace

int gemm_config_for(int64_t m, int64_t n) {
  if (m <= 32) return 0;
  const int64_t cl = gemm_cost<CfgLarge>(m, n), cm = gemm_cost<CfgMid>(m, n),
                cs = gemm_cost<CfgSmall>(m, n);
  if (cl <= cm && cl <= cs) return 3;
  return cm <= cs ? 2 : 1;
}

// Per-group scales: the 128 x 128 tile (its fp32 sums and int32 totals fit
// beside the accumulators).
int launch_gemm_mfma_group(const uint8_t* w, const int8_t* x, const float* x_scale,
                           const float* gs, float* y, int32_t* acc, int64_t m, int64_t n,
                           int64_t k, hipStream_t s) {
  using G = CfgSmall;
  const int MT = static_cast<int>(ceil_div(m, G::BM));
  const int NT = static_cast<int>(ceil_div(n, G::BN));
  const dim3 grid(static_cast<unsigned>(MT) * NT), block(G::THREADS);
  const WScale none{nullptr, 0.0f};
  if (k % kBK == 0)
    return launch(gemm_kernel<G, true, true>, grid, block, 0, s, w, x, x_scale, none, y, acc, m,
                  n, k, MT, NT, gs);
  return launch(gemm_kernel<G, false, true>, grid, block, 0, s, w, x, x_scale, none, y, acc, m,
                n, k, MT, NT, gs);
}

int launch_gemm_mfma(const uint8_t* w, const int8_t* x, const float* x_scale, WScale ws,
                     float* y, int32_t* acc, int64_t m, int64_t n, int64_t k, hipStream_t s) {
  switch (gemm_config_for(m, n)) {
    case 0: return launch_cfg<CfgSkinny>(w, x, x_scale, ws, y, acc, m, n, k, s);
    case 1: return launch_cfg<CfgSmall>(w, x, x_scale, ws, y, acc, m, n, k, s);
    case 2: return launch_cfg<CfgMid>(w, x, x_scale, ws, y, acc, m, n, k, s);
    default: return launch_cfg<CfgLarge>(w, x, x_scale, ws, y, acc, m, n, k, s);
  }
}

}  // namespace sherry
