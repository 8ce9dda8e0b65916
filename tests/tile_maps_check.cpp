// Host-side check of the workgroup -> tile maps of the product launches
// (xcd_remap, xcd_split_remap, deal_chunks, unrank_upper,
// unrank_strict_upper), compiled from the library's own header.  Prints
// "ok" and exits 0 when every property holds; prints the first failure and
// exits 1 otherwise.
#include <cstdio>
#include <vector>

#include "tile_mfma.hpp"

using namespace shp;

static int fail(const char* what, int a, int b, int c) {
  std::printf("FAIL %s (%d, %d, %d)\n", what, a, b, c);
  return 1;
}

int main() {
  // xcd_remap: a bijection on [0, n); XCD x (b % 8) gets a contiguous range,
  // in workgroup order
  for (int n = 0; n <= 300; ++n) {
    std::vector<int> seen(n, 0), last(8, -1);
    for (int b = 0; b < n; ++b) {
      const int l = xcd_remap(b, n);
      if (l < 0 || l >= n || seen[l]++) return fail("xcd_remap bijection", n, b, l);
      if (last[b & 7] >= 0 && l != last[b & 7] + 1) return fail("xcd_remap contiguous", n, b, l);
      last[b & 7] = l;
    }
  }
  // xcd_split_remap: over a grid of 8 (ceil((n1 + n2) / 8) + 1) workgroups,
  // every index of [0, n1 + n2) exactly once, -1 for the rest; each XCD runs
  // a contiguous range of the first part, then one of the second
  for (int n1 = 0; n1 <= 160; ++n1)
    for (int n2 = 0; n2 <= 90; ++n2) {
      const int grid = 8 * ((n1 + n2 + 7) / 8 + 1);
      std::vector<int> seen(n1 + n2, 0);
      for (int x = 0; x < 8; ++x) {
        int prev = -1;
        bool second = false;
        for (int b = x; b < grid; b += 8) {
          const int l = xcd_split_remap(b, n1, n2);
          if (l < 0) continue;
          if (l >= n1 + n2 || seen[l]++) return fail("xcd_split_remap bijection", n1, n2, b);
          if (l < n1 && second) return fail("xcd_split_remap first part after second", n1, n2, b);
          if (l >= n1 && !second) {
            second = true;
          } else if (prev >= 0 && l != prev + 1) {
            return fail("xcd_split_remap contiguous", n1, n2, b);
          }
          prev = l;
        }
      }
      for (int l = 0; l < n1 + n2; ++l)
        if (!seen[l]) return fail("xcd_split_remap missing", n1, n2, l);
      // with no second part it is xcd_remap over the first
      if (n2 == 0)
        for (int b = 0; b < n1; ++b)
          if (xcd_split_remap(b, n1, 0) != xcd_remap(b, n1)) return fail("xcd_split_remap n2 = 0", n1, b, 0);
    }
  // deal_chunks: a bijection on [0, 8 kDealChunk m)
  for (int m = 1; m <= 6; ++m) {
    const int n = 8 * kDealChunk * m;
    std::vector<int> seen(n, 0);
    for (int b = 0; b < n; ++b) {
      const int l = deal_chunks(b);
      if (l < 0 || l >= n || seen[l]++) return fail("deal_chunks bijection", m, b, l);
    }
  }
  // unrank_upper / unrank_strict_upper: row-major enumerations of the upper
  // (tj >= ti) and strictly upper (tj > ti) tiles of a T x T grid
  for (int T = 1; T <= 32; ++T) {
    int t = 0, s = 0;
    for (int i = 0; i < T; ++i)
      for (int j = i; j < T; ++j) {
        int ti, tj;
        unrank_upper(t++, T, ti, tj);
        if (ti != i || tj != j) return fail("unrank_upper", T, i, j);
        if (j > i) {
          unrank_strict_upper(s++, T, ti, tj);
          if (ti != i || tj != j) return fail("unrank_strict_upper", T, i, j);
        }
      }
  }
  std::printf("ok\n");
  return 0;
}
