// Host check of the query-tile orders the bf16 attention kernel walks (csrc/internal.h):
// plan_whole_tile and plan_split_tile must together enumerate every query tile exactly once,
// give each (batch, head) pair a run of split tiles at the end of its tiles (the same count
// to within one, the larger counts first), and number whole and split tiles pair by pair;
// xcd_remap must be a bijection that hands each XCD one contiguous range. Prints the number
// of violations and exits non-zero if there is any.
#include <cstdio>
#include <utility>
#include <vector>

#include "internal.h"

using refadapt::plan_split_tile;
using refadapt::plan_whole_tile;
using refadapt::xcd_remap;

int main() {
  long cases = 0, bad = 0;
  auto fail = [&](const char* what, int tiles, int nbh, int split) {
    if (bad++ < 10) std::printf("violation: %s (tiles per pair %d, pairs %d, split %d)\n", what, tiles, nbh, split);
  };
  auto fail_remap = [&](const char* what, int total) {
    if (bad++ < 10) std::printf("violation: %s (launch of %d tiles)\n", what, total);
  };
  // every plan with up to 70 query tiles per pair and up to 24 pairs, and a few wider launches
  std::vector<std::pair<int, int>> shapes;
  for (int tiles = 1; tiles <= 70; ++tiles)
    for (int nbh = 1; nbh <= 24; ++nbh) shapes.push_back({tiles, nbh});
  for (int nbh : {32, 48, 96})
    for (int tiles : {16, 65}) shapes.push_back({tiles, nbh});
  for (const auto& sh : shapes) {
    {
      const int tiles = sh.first, nbh = sh.second;
      const int total = tiles * nbh;
      for (int split = 0; split <= total; ++split) {
        ++cases;
        const int whole = total - split;
        std::vector<int> kind(total, 0);  // 1 whole, 2 split
        int last_pair = -1;
        for (int i = 0; i < whole; ++i) {
          const int t = plan_whole_tile(i, tiles, nbh, split);
          if (t < 0 || t >= total || kind[t] != 0) { fail("whole tile out of range or repeated", tiles, nbh, split); continue; }
          kind[t] = 1;
          if (t / tiles < last_pair) fail("whole tiles not numbered pair by pair", tiles, nbh, split);
          last_pair = t / tiles;
        }
        last_pair = -1;
        for (int s = 0; s < split; ++s) {
          const int t = plan_split_tile(s, tiles, nbh, split);
          if (t < 0 || t >= total || kind[t] != 0) { fail("split tile out of range or repeated", tiles, nbh, split); continue; }
          kind[t] = 2;
          if (t / tiles < last_pair) fail("split tiles not numbered pair by pair", tiles, nbh, split);
          last_pair = t / tiles;
        }
        const int q = split / nbh, r = split % nbh;
        for (int h = 0; h < nbh; ++h) {
          int n_split = 0;
          for (int k = 0; k < tiles; ++k) {
            const int v = kind[h * tiles + k];
            if (v == 0) fail("tile never enumerated", tiles, nbh, split);
            if (v == 2) ++n_split;
            else if (n_split > 0) fail("whole tile after a split tile of its pair", tiles, nbh, split);
          }
          if (n_split != q + (h < r ? 1 : 0)) fail("split tiles not spread evenly over the pairs", tiles, nbh, split);
        }
      }
    }
  }
  for (int total = 1; total <= 5000; ++total) {
    ++cases;
    std::vector<int> seen(total, 0);
    std::vector<int> lo(8, total), hi(8, -1), count(8, 0);
    for (int w = 0; w < total; ++w) {
      const int t = xcd_remap(w, total);
      if (t < 0 || t >= total || seen[t]++) { fail_remap("xcd_remap not a bijection", total); continue; }
      const int x = w & 7;
      lo[x] = t < lo[x] ? t : lo[x];
      hi[x] = t > hi[x] ? t : hi[x];
      ++count[x];
    }
    for (int x = 0; x < 8; ++x)
      if (count[x] > 0 && hi[x] - lo[x] + 1 != count[x]) fail_remap("an XCD's tiles are not contiguous", total);
  }
  std::printf("tile order cases %ld violations %ld\n", cases, bad);
  return bad != 0;
}
