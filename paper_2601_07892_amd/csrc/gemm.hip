// Prefill-path product (Eq. 2 at large M): the packed T tile is decoded once
// per workgroup into an int8 tile in LDS and multiplied with int8 MFMA.
//
// Per K-step of 128 (one unit column of the packed layout):
//  - X tile  BM x 128 int8: 16-byte global loads, written to LDS;
//  - T tile  BN x 128: BN/64 units of 1280 bytes; each thread decodes 32/TPR
//    codes of one row through the 32-entry table and writes int8 to LDS;
//  - 4 waves, each owning a (BM/WGM) x (BN/WGN) block of C made of 32x32
//    fragments, run v_mfma_i32_32x32x32_i8 over four 32-wide k slices.
// LDS rows are 128 bytes; 16-byte chunk c of row r lives at chunk c ^ (r&7),
// so the 8 rows read by any 8 lanes of a fragment load hit 8 distinct chunk
// positions (all 32 banks once).  Global loads for step s+1 are issued before
// the MFMAs of step s (register double buffering).
#include "sherry_internal.h"

namespace sherry {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));

constexpr int kGemmThreads = 256;
constexpr int kBK = 128;

template <int BM_, int BN_, int WGM_, int WGN_>
struct GemmCfg {
  static constexpr int BM = BM_, BN = BN_, WGM = WGM_, WGN = WGN_;
  static_assert(WGM * WGN == 4, "4 waves per workgroup");
  static constexpr int WM = BM / WGM, WN = BN / WGN;
  static_assert(WM % 32 == 0 && WN % 32 == 0, "32x32 fragments");
  static constexpr int FM = WM / 32, FN = WN / 32;
  static constexpr int XPT = BM * 8 / kGemmThreads;  // 16-byte X chunks per thread
  static_assert(XPT >= 1 && BM * 8 % kGemmThreads == 0, "X tile split");
  static constexpr int TPR = kGemmThreads / BN;  // threads decoding one T row
  static_assert(TPR >= 1 && TPR <= 4 && kGemmThreads % BN == 0, "T tile split");
  static constexpr int CPT = 32 / TPR;           // codes decoded per thread
  static constexpr int LDS_X = BM * kBK, LDS_W = BN * kBK;
};

__device__ __forceinline__ int swz(int row, int chunk) { return row * kBK + ((chunk ^ (row & 7)) << 4); }

// code*4 of code j (runtime j) of a container in d[0..4]
__device__ __forceinline__ uint32_t code_x4_rt(const uint32_t (&d)[5], int j) {
  const int bit = 5 * j, i = bit >> 5, off = bit & 31;
  const uint32_t lo = d[i];
  const uint32_t hi = (i < 4) ? d[i + 1] : d[i];
  const uint32_t prev = (i > 0) ? d[i - 1] : 0u;
  if (off >= 2) return __builtin_amdgcn_alignbit(hi, lo, off - 2) & 0x7Cu;
  return __builtin_amdgcn_alignbit(lo, prev, 30 + off) & 0x7Cu;
}

template <class G>
__global__ __launch_bounds__(kGemmThreads) void gemm_kernel(
    const uint8_t* __restrict__ w, const int8_t* __restrict__ x,
    const float* __restrict__ x_scale, float w_scale, float* __restrict__ y,
    int32_t* __restrict__ acc_out, int64_t M, int64_t N, int64_t K, int MT, int NT) {
  __shared__ uint32_t lut[32];
  __shared__ __attribute__((aligned(16))) int8_t xs[G::LDS_X];
  __shared__ __attribute__((aligned(16))) int8_t ws[G::LDS_W];

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

  // ---- per-thread load assignment ----
  // X: chunk q = tid + 256*v -> row q>>3, chunk q&7
  // T: row wrow = tid / TPR of the tile, part = tid % TPR
  const int wrow = tid / G::TPR, wpart = tid % G::TPR;
  const int64_t wunit_row = (n0 + wrow) / kTileRows;  // unit row of this T row
  const int wi = (int)((n0 + wrow) % kTileRows);
  const bool wrow_ok = wunit_row < R;

  uint4 xr[G::XPT];
  uint32_t wd[5];
  const bool k16 = (K % 16) == 0;

  auto load_step = [&](int64_t ks) {
    const int64_t kb = ks * kBK;
#pragma unroll
    for (int v = 0; v < G::XPT; ++v) {
      const int q = tid + kGemmThreads * v;
      const int row = q >> 3, ch = q & 7;
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
    if (wrow_ok) {
      const uint8_t* unit = w + (wunit_row * C + ks) * kUnitBytes;
      const uint4 h = *reinterpret_cast<const uint4*>(unit + 16 * wi);
      wd[0] = h.x;
      wd[1] = h.y;
      wd[2] = h.z;
      wd[3] = h.w;
      wd[4] = *reinterpret_cast<const uint32_t*>(unit + kHeadBytes + 4 * wi);
    } else {
      wd[0] = wd[1] = wd[2] = wd[3] = wd[4] = 0;
    }
  };

  auto store_step = [&]() {
#pragma unroll
    for (int v = 0; v < G::XPT; ++v) {
      const int q = tid + kGemmThreads * v;
      *reinterpret_cast<uint4*>(xs + swz(q >> 3, q & 7)) = xr[v];
    }
    // decode this thread's codes: CPT codes = CPT/4 chunks of 16 bytes
#pragma unroll
    for (int cc = 0; cc < G::CPT / 4; ++cc) {
      const int j0 = wpart * G::CPT + cc * 4;
      uint32_t q4[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const uint32_t a4 = code_x4_rt(wd, j0 + e);
        q4[e] = *reinterpret_cast<const uint32_t*>(reinterpret_cast<const char*>(lut) + a4);
      }
      *reinterpret_cast<uint4*>(ws + swz(wrow, j0 >> 2)) = make_uint4(q4[0], q4[1], q4[2], q4[3]);
    }
  };

  v16i acc[G::FM][G::FN];
#pragma unroll
  for (int a = 0; a < G::FM; ++a)
#pragma unroll
    for (int bb = 0; bb < G::FN; ++bb) acc[a][bb] = v16i{};

  load_step(0);
  __syncthreads();  // lut ready
  store_step();
  __syncthreads();

  const int frow = lane & 31, fhalf = lane >> 5;
  for (int64_t ks = 0; ks < C; ++ks) {
    if (ks + 1 < C) load_step(ks + 1);
#pragma unroll
    for (int t = 0; t < kBK / 32; ++t) {
      v4i af[G::FM], bf[G::FN];
#pragma unroll
      for (int a = 0; a < G::FM; ++a) {
        const int row = wr * G::WM + a * 32 + frow;
        af[a] = *reinterpret_cast<const v4i*>(xs + swz(row, 2 * t + fhalf));
      }
#pragma unroll
      for (int bb = 0; bb < G::FN; ++bb) {
        const int row = wc * G::WN + bb * 32 + frow;
        bf[bb] = *reinterpret_cast<const v4i*>(ws + swz(row, 2 * t + fhalf));
      }
#pragma unroll
      for (int a = 0; a < G::FM; ++a)
#pragma unroll
        for (int bb = 0; bb < G::FN; ++bb)
          acc[a][bb] = __builtin_amdgcn_mfma_i32_32x32x32_i8(af[a], bf[bb], acc[a][bb], 0, 0, 0);
    }
    __syncthreads();
    if (ks + 1 < C) {
      store_step();
      __syncthreads();
    }
  }

  // ---- epilogue: lane holds C[i][j] with j = lane%32 and
  //      i = 8*(r/4) + 4*(lane/32) + r%4 for accumulator element r
#pragma unroll
  for (int a = 0; a < G::FM; ++a) {
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int64_t gm = m0 + wr * G::WM + a * 32 + 8 * (r >> 2) + 4 * fhalf + (r & 3);
      if (gm >= M) continue;
      const float s = x_scale[gm] * w_scale;
#pragma unroll
      for (int bb = 0; bb < G::FN; ++bb) {
        const int64_t gn = n0 + wc * G::WN + bb * 32 + frow;
        if (gn >= N) continue;
        const int32_t v = acc[a][bb][r];
        y[gm * N + gn] = static_cast<float>(v) * s;
        if (acc_out) acc_out[gm * N + gn] = v;
      }
    }
  }
}

template <class G>
int launch_cfg(const uint8_t* w, const int8_t* x, const float* x_scale, float w_scale,
               float* y, int32_t* acc, int64_t m, int64_t n, int64_t k, hipStream_t s) {
  const int MT = static_cast<int>(ceil_div(m, G::BM));
  const int NT = static_cast<int>(ceil_div(n, G::BN));
  return launch(gemm_kernel<G>, dim3(static_cast<unsigned>(MT) * NT), dim3(kGemmThreads),
                     0, s, w, x, x_scale, w_scale, y, acc, m, n, k, MT, NT);
}

using CfgLarge = GemmCfg<256, 256, 2, 2>;  // wave tile 128 x 128
using CfgMid = GemmCfg<128, 256, 2, 2>;    // wave tile 64 x 128
using CfgSkinny = GemmCfg<32, 256, 1, 4>;  // wave tile 32 x 64

}  // namespace

int launch_gemm_mfma(const uint8_t* w, const int8_t* x, const float* x_scale, float w_scale,
                     float* y, int32_t* acc, int64_t m, int64_t n, int64_t k, hipStream_t s) {
  if (m <= 32) return launch_cfg<CfgSkinny>(w, x, x_scale, w_scale, y, acc, m, n, k, s);
  const int64_t big_tiles = ceil_div(m, 256) * ceil_div(n, 256);
  if (big_tiles >= 256) return launch_cfg<CfgLarge>(w, x, x_scale, w_scale, y, acc, m, n, k, s);
  return launch_cfg<CfgMid>(w, x, x_scale, w_scale, y, acc, m, n, k, s);
}

}  // namespace sherry
