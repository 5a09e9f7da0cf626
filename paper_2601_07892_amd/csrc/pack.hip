// Offline packing (Appendix A, offline phase): host code.
//
// sherry_pack turns a ternary 3:4 matrix into the 5-bit tiled layout that the
// device products stream; sherry_unpack is its exact inverse.  sherry_pack_il
// writes the same codes lane-interleaved for the matrix-core products.
// sherry_pack2 and sherry_pack3 write the two comparison layouts (2 bits per
// weight, and three weights per 5-bit code).  Layouts are defined in
// sherry.h.
#include <algorithm>
#include <atomic>
#include <cstring>
#include <thread>
#include <vector>

#include "sherry_internal.h"

namespace sherry {
namespace {

// Code of one block, or -1 if it does not hold exactly one zero and three
// values in {-1, +1} (Eq. 3).
inline int encode_block(const int8_t* w) {
  int z = -1;
  uint32_t neg = 0;  // bit p set when weight p is -1
  for (int p = 0; p < 4; ++p) {
    const int v = w[p];
    if (v == 0) {
      if (z >= 0) return -1;
      z = p;
    } else if (v == -1) {
      neg |= 1u << p;
    } else if (v != 1) {
      return -1;
    }
  }
  if (z < 0) return -1;
  // drop the zero's position: sign bits of the non-zeros, ascending
  const uint32_t below = neg & ((1u << z) - 1u);
  const uint32_t above = neg >> (z + 1);
  return static_cast<int>(static_cast<uint32_t>(z) | ((below | (above << z)) << 2));
}

unsigned worker_count(int64_t jobs) {
  unsigned hw = std::thread::hardware_concurrency();
  if (hw == 0) hw = 4;
  hw = std::min(hw, 32u);
  return static_cast<unsigned>(std::max<int64_t>(1, std::min<int64_t>(hw, jobs)));
}

// Runs fn(begin, end) over [0, jobs) split into contiguous ranges.
template <class Fn>
void parallel_ranges(int64_t jobs, Fn fn) {
  const unsigned nt = worker_count(jobs);
  if (nt <= 1) {
    fn(int64_t(0), jobs);
    return;
  }
  std::vector<std::thread> th;
  th.reserve(nt);
  for (unsigned t = 0; t < nt; ++t) {
    const int64_t b = jobs * t / nt, e = jobs * (t + 1) / nt;
    th.emplace_back([=] { fn(b, e); });
  }
  for (auto& x : th) x.join();
}

// Packs the 32 codes of one row container into 16 head bytes + 4 tail bytes.
inline void put_container(const uint32_t* codes, uint8_t* head, uint8_t* tail) {
  uint64_t lo = 0, mid = 0;
  uint32_t hi = 0;
  for (int j = 0; j < 32; ++j) {
    const uint64_t c = codes[j];
    const int b = 5 * j;
    if (b + 5 <= 64) {
      lo |= c << b;
    } else if (b < 64) {  // straddles bit 64
      lo |= c << b;
      mid |= c >> (64 - b);
    } else if (b + 5 <= 128) {
      mid |= c << (b - 64);
    } else if (b < 128) {  // straddles bit 128
      mid |= c << (b - 64);
      hi |= static_cast<uint32_t>(c >> (128 - b));
    } else {
      hi |= static_cast<uint32_t>(c << (b - 128));
    }
  }
  std::memcpy(head, &lo, 8);
  std::memcpy(head + 8, &mid, 8);
  std::memcpy(tail, &hi, 4);
}

inline void get_container(const uint8_t* head, const uint8_t* tail, uint32_t* codes) {
  uint64_t lo, mid;
  uint32_t hi;
  std::memcpy(&lo, head, 8);
  std::memcpy(&mid, head + 8, 8);
  std::memcpy(&hi, tail, 4);
  for (int j = 0; j < 32; ++j) {
    const int b = 5 * j;
    uint64_t v;
    if (b + 5 <= 64) v = lo >> b;
    else if (b < 64) v = (lo >> b) | (mid << (64 - b));
    else if (b + 5 <= 128) v = mid >> (b - 64);
    else if (b < 128) v = (mid >> (b - 64)) | (static_cast<uint64_t>(hi) << (128 - b));
    else v = hi >> (b - 128);
    codes[j] = static_cast<uint32_t>(v & 31u);
  }
}

// Lane-interleaved units: the container of lane l = 16b + t holds, as code
// j = 4(2g + p) + c, the code of row 16g + t and block 16p + 4b + c of the
// unit (g, b = 0..3, p = 0..1, c = 0..3).  il_source gives, for (l, j), the
// row and block of the unit that the tiled layout keeps in lane `row`, code
// `block`.
inline void il_source(int l, int j, int* row, int* block) {
  const int b = l >> 4, t = l & 15;
  const int g = j >> 3, p = (j >> 2) & 1, c = j & 3;
  *row = 16 * g + t;
  *block = 16 * p + 4 * b + c;
}

}  // namespace
}  // namespace sherry

using namespace sherry;

extern "C" size_t sherry_packed_bytes(int64_t n, int64_t k) {
  if (n < 1 || k < 1 || k % 4 != 0 || n > SHERRY_MAX_N || k > SHERRY_MAX_K) return 0;
  return static_cast<size_t>(ceil_div(n, kTileRows) * kTileRows) *
         static_cast<size_t>(ceil_div(k, kTileK) * kTileK) * 5 / 32;
}

extern "C" int sherry_pack(const int8_t* t, int64_t n, int64_t k, uint8_t* out,
                           size_t out_bytes, int64_t* bad_block) {
  if (!t || !out) return SHERRY_E_INVALID;
  const size_t need = sherry_packed_bytes(n, k);
  if (need == 0) return SHERRY_E_SHAPE;
  if (out_bytes < need) return SHERRY_E_BUFSIZE;
  const int64_t R = ceil_div(n, kTileRows), C = ceil_div(k, kTileK);
  const int64_t nb = k / 4;
  std::atomic<int64_t> first_bad{INT64_MAX};
  parallel_ranges(R, [&](int64_t r0, int64_t r1) {
    uint32_t codes[32];
    for (int64_t r = r0; r < r1; ++r) {
      for (int64_t c = 0; c < C; ++c) {
        uint8_t* unit = out + static_cast<size_t>(r * C + c) * kUnitBytes;
        for (int i = 0; i < kTileRows; ++i) {
          const int64_t row = r * kTileRows + i;
          for (int j = 0; j < 32; ++j) {
            const int64_t b = c * 32 + j;
            int code = 0;
            if (row < n && b < nb) {
              code = encode_block(t + row * k + 4 * b);
              if (code < 0) {
                const int64_t flat = row * nb + b;
                int64_t cur = first_bad.load();
                while (flat < cur && !first_bad.compare_exchange_weak(cur, flat)) {
                }
                code = 0;
              }
            }
            codes[j] = static_cast<uint32_t>(code);
          }
          put_container(codes, unit + 16 * i, unit + kHeadBytes + 4 * i);
        }
      }
    }
  });
  if (first_bad.load() != INT64_MAX) {
    if (bad_block) *bad_block = first_bad.load();
    return SHERRY_E_NOT_3_4;
  }
  return SHERRY_OK;
}

extern "C" int sherry_unpack(const uint8_t* packed, size_t packed_bytes, int64_t n,
                             int64_t k, int8_t* t_out) {
  if (!packed || !t_out) return SHERRY_E_INVALID;
  const size_t need = sherry_packed_bytes(n, k);
  if (need == 0) return SHERRY_E_SHAPE;
  if (packed_bytes < need) return SHERRY_E_BUFSIZE;
  const int64_t R = ceil_div(n, kTileRows), C = ceil_div(k, kTileK);
  const int64_t nb = k / 4;
  parallel_ranges(R, [&](int64_t r0, int64_t r1) {
    uint32_t codes[32];
    for (int64_t r = r0; r < r1; ++r) {
      for (int64_t c = 0; c < C; ++c) {
        const uint8_t* unit = packed + static_cast<size_t>(r * C + c) * kUnitBytes;
        for (int i = 0; i < kTileRows; ++i) {
          const int64_t row = r * kTileRows + i;
          if (row >= n) break;
          get_container(unit + 16 * i, unit + kHeadBytes + 4 * i, codes);
          for (int j = 0; j < 32; ++j) {
            const int64_t b = c * 32 + j;
            if (b >= nb) break;
            const uint32_t word = decode_word(codes[j]);
            for (int p = 0; p < 4; ++p)
              t_out[row * k + 4 * b + p] = static_cast<int8_t>((word >> (8 * p)) & 0xFF);
          }
        }
      }
    }
  });
  return SHERRY_OK;
}

extern "C" size_t sherry_packed2_bytes(int64_t n, int64_t k) {
  if (n < 1 || k < 1 || k % 4 != 0 || n > SHERRY_MAX_N || k > SHERRY_MAX_K) return 0;
  return static_cast<size_t>(ceil_div(n, kTileRows) * kTileRows) *
         static_cast<size_t>(ceil_div(k, kTileK2) * kTileK2) / 4;
}

extern "C" int sherry_pack2(const int8_t* t, int64_t n, int64_t k, uint8_t* out,
                            size_t out_bytes, int64_t* bad_index) {
  if (!t || !out) return SHERRY_E_INVALID;
  const size_t need = sherry_packed2_bytes(n, k);
  if (need == 0) return SHERRY_E_SHAPE;
  if (out_bytes < need) return SHERRY_E_BUFSIZE;
  const int64_t R = ceil_div(n, kTileRows), C = ceil_div(k, kTileK2);
  std::atomic<int64_t> first_bad{INT64_MAX};
  parallel_ranges(R, [&](int64_t r0, int64_t r1) {
    for (int64_t r = r0; r < r1; ++r) {
      for (int64_t c = 0; c < C; ++c) {
        uint8_t* unit = out + static_cast<size_t>(r * C + c) * kUnit2Bytes;
        for (int i = 0; i < kTileRows; ++i) {
          const int64_t row = r * kTileRows + i;
          // every field starts as weight 0 (value 1)
          uint32_t word[4] = {0x55555555u, 0x55555555u, 0x55555555u, 0x55555555u};
          if (row < n) {
            for (int u = 0; u < kTileK2; ++u) {
              const int64_t kk = c * kTileK2 + u;
              if (kk >= k) break;
              const int v = t[row * k + kk];
              if (v < -1 || v > 1) {
                const int64_t flat = row * k + kk;
                int64_t cur = first_bad.load();
                while (flat < cur && !first_bad.compare_exchange_weak(cur, flat)) {
                }
                continue;
              }
              // u = 16 wd + 4 j + p: word wd, byte p, bits [2j, 2j + 2)
              const int wd = u >> 4, sh = 8 * (u & 3) + 2 * ((u >> 2) & 3);
              word[wd] = (word[wd] & ~(3u << sh)) | (static_cast<uint32_t>(v + 1) << sh);
            }
          }
          std::memcpy(unit + 16 * i, word, 16);
        }
      }
    }
  });
  if (first_bad.load() != INT64_MAX) {
    if (bad_index) *bad_index = first_bad.load();
    return SHERRY_E_INVALID;
  }
  return SHERRY_OK;
}

// ---- 1.67-bit comparison layout: three weights per 5-bit code ------------

extern "C" size_t sherry_packed3_bytes(int64_t n, int64_t k) {
  if (n < 1 || k < 1 || n > SHERRY_MAX_N || k > SHERRY_MAX_K) return 0;
  return static_cast<size_t>(ceil_div(n, kTileRows) * kTileRows) *
         static_cast<size_t>(ceil_div(k, kTileK3)) * kUnitBytes / kTileRows;
}

extern "C" int sherry_pack3(const int8_t* t, int64_t n, int64_t k, uint8_t* out,
                            size_t out_bytes, int64_t* bad_index) {
  if (!t || !out) return SHERRY_E_INVALID;
  const size_t need = sherry_packed3_bytes(n, k);
  if (need == 0) return SHERRY_E_SHAPE;
  if (out_bytes < need) return SHERRY_E_BUFSIZE;
  const int64_t R = ceil_div(n, kTileRows), C = ceil_div(k, kTileK3);
  std::atomic<int64_t> first_bad{INT64_MAX};
  parallel_ranges(R, [&](int64_t r0, int64_t r1) {
    uint32_t codes[32];
    for (int64_t r = r0; r < r1; ++r) {
      for (int64_t c = 0; c < C; ++c) {
        uint8_t* unit = out + static_cast<size_t>(r * C + c) * kUnitBytes;
        for (int i = 0; i < kTileRows; ++i) {
          const int64_t row = r * kTileRows + i;
          for (int j = 0; j < 32; ++j) {
            // base-3 digits w + 1, least significant first; weights past k
            // and rows past n are 0 (digit 1)
            uint32_t code = 0, scale = 1;
            for (int q = 0; q < 3; ++q, scale *= 3) {
              const int64_t kk = c * kTileK3 + 3 * j + q;
              int v = 0;
              if (row < n && kk < k) {
                v = t[row * k + kk];
                if (v < -1 || v > 1) {
                  const int64_t flat = row * k + kk;
                  int64_t cur = first_bad.load();
                  while (flat < cur && !first_bad.compare_exchange_weak(cur, flat)) {
                  }
                  v = 0;
                }
              }
              code += static_cast<uint32_t>(v + 1) * scale;
            }
            codes[j] = code;
          }
          put_container(codes, unit + 16 * i, unit + kHeadBytes + 4 * i);
        }
      }
    }
  });
  if (first_bad.load() != INT64_MAX) {
    if (bad_index) *bad_index = first_bad.load();
    return SHERRY_E_INVALID;
  }
  return SHERRY_OK;
}

extern "C" int sherry_unpack3(const uint8_t* packed, size_t packed_bytes, int64_t n,
                              int64_t k, int8_t* t_out) {
  if (!packed || !t_out) return SHERRY_E_INVALID;
  const size_t need = sherry_packed3_bytes(n, k);
  if (need == 0) return SHERRY_E_SHAPE;
  if (packed_bytes < need) return SHERRY_E_BUFSIZE;
  const int64_t R = ceil_div(n, kTileRows), C = ceil_div(k, kTileK3);
  std::atomic<bool> bad{false};
  parallel_ranges(R, [&](int64_t r0, int64_t r1) {
    uint32_t codes[32];
    for (int64_t r = r0; r < r1; ++r) {
      for (int64_t c = 0; c < C; ++c) {
        const uint8_t* unit = packed + static_cast<size_t>(r * C + c) * kUnitBytes;
        for (int i = 0; i < kTileRows; ++i) {
          const int64_t row = r * kTileRows + i;
          if (row >= n) break;
          get_container(unit + 16 * i, unit + kHeadBytes + 4 * i, codes);
          for (int j = 0; j < 32; ++j) {
            uint32_t code = codes[j];
            const int64_t kk0 = c * kTileK3 + 3 * j;
            if (kk0 >= k) break;
            if (code > 26) bad.store(true);
            for (int q = 0; q < 3; ++q, code /= 3)
              if (kk0 + q < k) t_out[row * k + kk0 + q] = static_cast<int8_t>(int(code % 3) - 1);
          }
        }
      }
    }
  });
  return bad.load() ? SHERRY_E_INVALID : SHERRY_OK;
}

extern "C" int sherry_pack_il(const int8_t* t, int64_t n, int64_t k, uint8_t* out,
                              size_t out_bytes, int64_t* bad_block) {
  // the tiled units first, then each unit's codes moved to their lanes
  const int st = sherry_pack(t, n, k, out, out_bytes, bad_block);
  if (st != SHERRY_OK) return st;
  const int64_t units = ceil_div(n, kTileRows) * ceil_div(k, kTileK);
  parallel_ranges(units, [&](int64_t u0, int64_t u1) {
    uint32_t tiled[kTileRows][32], codes[32];
    for (int64_t u = u0; u < u1; ++u) {
      uint8_t* unit = out + static_cast<size_t>(u) * kUnitBytes;
      for (int i = 0; i < kTileRows; ++i)
        get_container(unit + 16 * i, unit + kHeadBytes + 4 * i, tiled[i]);
      for (int l = 0; l < kTileRows; ++l) {
        for (int j = 0; j < 32; ++j) {
          int row, block;
          il_source(l, j, &row, &block);
          codes[j] = tiled[row][block];
        }
        put_container(codes, unit + 16 * l, unit + kHeadBytes + 4 * l);
      }
    }
  });
  return SHERRY_OK;
}

extern "C" int sherry_unpack_il(const uint8_t* packed, size_t packed_bytes, int64_t n,
                                int64_t k, int8_t* t_out) {
  if (!packed || !t_out) return SHERRY_E_INVALID;
  const size_t need = sherry_packed_bytes(n, k);
  if (need == 0) return SHERRY_E_SHAPE;
  if (packed_bytes < need) return SHERRY_E_BUFSIZE;
  // back to tiled units in a copy, then the tiled unpacker
  std::vector<uint8_t> tiled(need);
  const int64_t units = ceil_div(n, kTileRows) * ceil_div(k, kTileK);
  parallel_ranges(units, [&](int64_t u0, int64_t u1) {
    uint32_t il[kTileRows][32];
    for (int64_t u = u0; u < u1; ++u) {
      const uint8_t* src = packed + static_cast<size_t>(u) * kUnitBytes;
      uint8_t* dst = tiled.data() + static_cast<size_t>(u) * kUnitBytes;
      for (int l = 0; l < kTileRows; ++l)
        get_container(src + 16 * l, src + kHeadBytes + 4 * l, il[l]);
      uint32_t rows[kTileRows][32];
      for (int l = 0; l < kTileRows; ++l) {
        for (int j = 0; j < 32; ++j) {
          int row, block;
          il_source(l, j, &row, &block);
          rows[row][block] = il[l][j];
        }
      }
      for (int i = 0; i < kTileRows; ++i)
        put_container(rows[i], dst + 16 * i, dst + kHeadBytes + 4 * i);
    }
  });
  return sherry_unpack(tiled.data(), need, n, k, t_out);
}

