// Exercises the library's host packers (sherry_pack, sherry_unpack,
// sherry_pack2) on ragged shapes, built with AddressSanitizer and
// UndefinedBehaviorSanitizer on the host side only (no GPU call is made).
// Exit status 0 when every round trip and rejection holds.
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <vector>

#include "sherry.h"

namespace {

uint64_t g_state = 0x243F6A8885A308D3ull;
uint64_t next_u64() {  // SplitMix64
  uint64_t z = (g_state += 0x9E3779B97F4A7C15ull);
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

// A random 3:4 block: zero at a random position, random signs elsewhere.
void block(int8_t* w) {
  const uint64_t r = next_u64();
  const int z = static_cast<int>(r & 3);
  for (int p = 0; p < 4; ++p) w[p] = (p == z) ? 0 : (((r >> (2 + p)) & 1) ? -1 : 1);
}

bool one_shape(int64_t n, int64_t k) {
  std::vector<int8_t> t(static_cast<size_t>(n * k)), back(t.size());
  for (int64_t b = 0; b < n * k / 4; ++b) block(&t[static_cast<size_t>(4 * b)]);
  const size_t nb = sherry_packed_bytes(n, k);
  std::vector<uint8_t> p(nb);
  int64_t bad = -5;
  if (sherry_pack(t.data(), n, k, p.data(), nb, &bad) != SHERRY_OK || bad != -5) return false;
  if (sherry_unpack(p.data(), nb, n, k, back.data()) != SHERRY_OK || back != t) return false;
  // one byte short is refused, nothing is written past the buffer
  if (sherry_pack(t.data(), n, k, p.data(), nb - 1, nullptr) != SHERRY_E_BUFSIZE) return false;
  const size_t nb2 = sherry_packed2_bytes(n, k);
  std::vector<uint8_t> p2(nb2);
  if (sherry_pack2(t.data(), n, k, p2.data(), nb2, nullptr) != SHERRY_OK) return false;
  // a block with two zeros in the last row: rejected with its flat index
  std::vector<int8_t> t3 = t;
  const int64_t blk = n * (k / 4) - 1;
  std::memset(&t3[static_cast<size_t>(4 * blk)], 0, 2);
  t3[static_cast<size_t>(4 * blk + 2)] = 1;
  t3[static_cast<size_t>(4 * blk + 3)] = -1;
  if (sherry_pack(t3.data(), n, k, p.data(), nb, &bad) != SHERRY_E_NOT_3_4 || bad != blk)
    return false;
  return true;
}

}  // namespace

int main() {
  const int64_t shapes[][2] = {{1, 4}, {65, 132}, {130, 516}, {64, 2048}, {7, 12}, {200, 1028},
                               {3, 4100}};
  for (const auto& s : shapes) {
    if (!one_shape(s[0], s[1])) {
      std::fprintf(stderr, "packer check failed for n=%lld k=%lld\n",
                   static_cast<long long>(s[0]), static_cast<long long>(s[1]));
      return 1;
    }
  }
  std::puts("packer sanitizer driver: ok");
  return 0;
}
