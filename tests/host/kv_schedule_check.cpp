// Host check of the key-stationary backward's work schedule (kv_chunk_rows,
// kv_unit, kv_units, kv_masked_steps in basp_internal.hpp), for many sequence
// lengths, at the chunk the library picks and at every other chunk size it
// could take:
//  * every (key tile, row chunk) pair with rows to do is some unit exactly
//    once, and units past the last key tile or with empty rows do nothing;
//  * the full units come before the diagonal ones, and the diagonal units
//    run longest first (within a chunk; overall when S fills whole chunks);
//  * the first chunk a key tile writes is chunk k0 / C (the
//    reduction starts there);
//  * the steps of a unit after its masked ones start at or after the last
//    key of the tile, so no wave's keys need a mask there, and each masked
//    step does overlap the tile's keys.
// Prints the number of sequence lengths checked; exits 1 at the first
// failure.
#include <stdio.h>

#include <algorithm>
#include <map>
#include <utility>
#include <vector>

#include "../../paper_2609_03151_amd/csrc/basp_internal.hpp"

using namespace basp;

static int fail(const char *what, int S, int a, int b) {
  printf("FAIL %s: S=%d (%d, %d)\n", what, S, a, b);
  return 1;
}

int main() {
  std::vector<int> lengths = {1, 2, 63, 64, 65, 127, 128, 129, 255, 256, 300, 1000, 2047, 2048,
                              2049, 2500, 4095, 4096, 4097, 6000, 8192, 16384, 32768, 65536,
                              131072, 131073, 200000, 262144, 524289};
  for (int S = 64; S <= 40000; S += 997) lengths.push_back(S);
  const int step_rows = 64;
  int checked = 0;
  for (int S : lengths) {
    if ((S + kv_chunk_rows(S) - 1) / kv_chunk_rows(S) > kKvMaxChunks)
      return fail("more row chunks than the cap", S, kv_chunk_rows(S), 0);
    for (int C : {kv_chunk_rows(S), 2048, 4096, 8192, 128, 384}) {
      if (S > 131072 && C != kv_chunk_rows(S)) continue;  // long ones: the library's chunk only
      if (C % kKvKeys != 0) return fail("chunk not a multiple of the key tile", S, C, 0);
      const int T = C / kKvKeys;
      const int nch = (S + C - 1) / C;
      const int ktiles = (S + kKvKeys - 1) / kKvKeys;
      std::map<std::pair<int, int>, int> seen;
      std::map<int, int> first_chunk;
      bool in_diag = false;
      long last_len = -1;
      std::map<int, long> last_len_ch;
      for (int u = 0; u < kv_units(nch, T); ++u) {
        int kt, ch;
        kv_unit(u, nch, T, kt, ch);
        if (kt < 0 || ch < 0 || ch >= nch) return fail("unit out of range", S, kt, ch);
        if (kt >= ktiles) continue;
        const int k0 = kt * kKvKeys;
        const int r_lo = std::max(k0, ch * C);
        const int r_hi = std::min(S, (ch + 1) * C);
        if (r_lo >= r_hi) continue;
        if (++seen[{kt, ch}] > 1) return fail("pair twice", S, kt, ch);
        const bool full = r_lo == ch * C;
        if (full && in_diag) return fail("full unit after a diagonal one", S, kt, ch);
        if (!full) {  // longest first within a chunk, and overall when every chunk is whole
          const long len = r_hi - r_lo;
          if (last_len_ch.count(ch) && len > last_len_ch[ch])
            return fail("diagonal units of a chunk not longest first", S, kt, ch);
          if (S % C == 0 && in_diag && len > last_len)
            return fail("diagonal units not longest first", S, kt, ch);
          in_diag = true;
          last_len = len;
          last_len_ch[ch] = len;
        }
        if (!first_chunk.count(kt) || ch < first_chunk[kt]) first_chunk[kt] = ch;
        // masked steps
        const int steps = (r_hi - r_lo + step_rows - 1) / step_rows;
        const int nm = kv_masked_steps(k0, r_lo, steps, step_rows);
        for (int t = 0; t < steps; ++t) {
          const int i0 = r_lo + t * step_rows;
          for (int w = 0; w < kKvKeys / 32; ++w) {
            const int wk0 = k0 + 32 * w;
            const bool needs_mask = i0 < wk0 + 31;  // some row of the step precedes a key
            if (t >= nm && needs_mask) return fail("unmasked step needs a mask", S, kt, t);
          }
          if (t < nm && !(i0 < k0 + kKvKeys - 1)) return fail("masked step clear of the keys", S, kt, t);
        }
      }
      // coverage: every pair with rows is present
      for (int kt = 0; kt < ktiles; ++kt) {
        const int k0 = kt * kKvKeys;
        for (int ch = 0; ch < nch; ++ch) {
          const int r_lo = std::max(k0, ch * C);
          const int r_hi = std::min(S, (ch + 1) * C);
          if (r_lo < r_hi && !seen.count({kt, ch})) return fail("pair missing", S, kt, ch);
        }
        if (first_chunk[kt] != k0 / C) return fail("first chunk", S, kt, first_chunk[kt]);
      }
      ++checked;
    }
  }
  printf("kv schedule ok %d\n", checked);
  return 0;
}
