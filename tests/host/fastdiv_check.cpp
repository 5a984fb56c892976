// Host check of the multiply-high division every kernel of libbasp uses for
// row -> (buffer, row in buffer) and vector -> (row, column): q = n / d for
// many divisors and dividends, against the hardware divide.  Prints the
// number of (d, n) pairs checked; exits 1 at the first mismatch.
#include <stdint.h>
#include <stdio.h>

#include <vector>

#include "../../paper_2609_03151_amd/csrc/basp_internal.hpp"

static uint64_t state = 0x9E3779B97F4A7C15ull;
static uint32_t next_u32() {  // xorshift64*
  state ^= state >> 12;
  state ^= state << 25;
  state ^= state >> 27;
  return (uint32_t)((state * 0x2545F4914F6CDD1Dull) >> 32);
}

int main() {
  std::vector<uint32_t> divisors;
  for (uint32_t d = 1; d <= 5000; ++d) divisors.push_back(d);
  for (int k = 1; k < 32; ++k) {
    const uint32_t p = 1u << k;
    divisors.push_back(p - 1);
    divisors.push_back(p);
    divisors.push_back(p + 1);
  }
  const uint32_t shard_rows[] = {256, 768, 1024, 2560, 5461, 8192, 10923, 16384, 32768, 131072};
  for (uint32_t d : shard_rows) divisors.push_back(d);
  for (int i = 0; i < 2000; ++i) divisors.push_back(1 + next_u32() % 0x7FFFFFFFu);
  divisors.push_back(0x7FFFFFFFu);
  divisors.push_back(0x80000000u);
  divisors.push_back(0xFFFFFFFFu);

  unsigned long long checked = 0;
  for (uint32_t d : divisors) {
    const basp::FastDiv f = basp::FastDiv::make(d);
    std::vector<uint32_t> ns = {0u, 1u, d - 1, d, d + 1, 2 * d - 1, 2 * d, 0x7FFFFFFFu,
                                0x80000000u, 0xFFFFFFFEu, 0xFFFFFFFFu};
    for (int i = 0; i < 64; ++i) ns.push_back(next_u32());
    for (int i = 0; i < 16; ++i) {  // multiples and their neighbours
      const uint64_t k = next_u32() % (0xFFFFFFFFull / d + 1);
      const uint64_t x = k * d;
      for (int e = -1; e <= 1; ++e) {
        const int64_t y = (int64_t)x + e;
        if (y >= 0 && y <= 0xFFFFFFFFll) ns.push_back((uint32_t)y);
      }
    }
    for (uint32_t n : ns) {
      if (f.div(n) != n / d) {
        printf("MISMATCH d=%u n=%u got=%u want=%u\n", d, n, f.div(n), n / d);
        return 1;
      }
      ++checked;
    }
  }
  printf("fastdiv ok %llu\n", checked);
  return 0;
}
