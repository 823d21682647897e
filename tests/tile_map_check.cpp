// Host build of the product kernel's tile placement (gemm.h): checks the
// spread row order, whole and whole-rounds launches plus K-split tails, and
// that the dealt groups keep the XCDs on the same column tiles.
// Prints "ok" and exits 0, or names the first failing case and exits 1.
#include <algorithm>
#include <cstdio>
#include <map>
#include <set>
#include <utility>
#include <vector>

#include "gemm.h"

using namespace pspo;

static int fail(const char* what, int a, int b, int c) {
  std::printf("FAIL %s %d %d %d\n", what, a, b, c);
  return 1;
}

// spread_row_tile: a bijection on [0, T) whose first s tiles appear in order
static int check_spread() {
  for (int T = 1; T <= 400; ++T)
    for (int s = 0; s <= T; s += (T > 40 ? 7 : 1)) {
      std::vector<int> seen(T, 0);
      int next_kept = 0;
      for (int l = 0; l < T; ++l) {
        const int p = spread_row_tile(l, s, T);
        if (p < 0 || p >= T || seen[p]++) return fail("spread bijection", T, s, l);
        if (p < s && p != next_kept++) return fail("spread order", T, s, l);
      }
    }
  return 0;
}

// whole launch, and whole rounds + K-split tail: every tile once, each tail
// tile's K parts partition [0, nk), slabs unique and below 8 x kTailSlots
static int check_launches(int tiles_m, int tiles_n, int M, int N, int nk) {
  const int grid = (tiles_m * tiles_n + kNumXcd - 1) / kNumXcd * kNumXcd;
  const TileGrid tg = tile_grid(tiles_m, tiles_n, M, N);
  std::set<std::pair<int, int>> whole;
  for (int bid = 0; bid < grid; ++bid) {
    int tm, tn;
    if (map_tile_at(bid, tiles_m, tiles_n, M, N, tm, tn, 0, false))
      if (!whole.insert({tm, tn}).second) return fail("whole duplicate", tiles_m, tiles_n, bid);
  }
  if ((int)whole.size() != tg.total) return fail("whole coverage", tiles_m, tiles_n, (int)whole.size());
  std::map<std::pair<int, int>, std::vector<std::pair<int, int>>> parts;
  for (int bid = 0; bid < grid; ++bid) {
    int tm, tn;
    if (map_tile_at(bid, tiles_m, tiles_n, M, N, tm, tn, 0, true)) parts[{tm, tn}].push_back({0, nk});
  }
  for (int bid = 0; bid < kNumXcd * kTailSlots; ++bid) {
    int tm, tn, kb, ke;
    if (!map_tail(tg, bid, nk, tm, tn, kb, ke)) continue;
    if (nk > 0 && ke <= kb) return fail("empty K part", tiles_m, tiles_n, bid);
    parts[{tm, tn}].push_back({kb, ke});
  }
  if ((int)parts.size() != tg.total) return fail("rounds + tail coverage", tiles_m, tiles_n, (int)parts.size());
  for (auto& kv : parts) {
    auto& v = kv.second;
    std::sort(v.begin(), v.end());
    int pos = 0;
    for (auto& r : v) {
      if (r.first != pos) return fail("K partition", kv.first.first, kv.first.second, r.first);
      pos = r.second;
    }
    if (pos != nk) return fail("K end", kv.first.first, kv.first.second, pos);
  }
  int sum = 0;
  for (int x = 0; x < kNumXcd; ++x) {
    const int c = xcd_count(tg, x);
    sum += c;
    if (c > tg.per_xcd) return fail("positions per XCD", tiles_m, tiles_n, c);
    const int r = c - tg.per_xcd / 32 * 32;
    if (r > 31) return fail("tail tiles per XCD", tiles_m, tiles_n, r);
  }
  if (sum != tg.total) return fail("positions of all XCDs", tiles_m, tiles_n, sum);
  // the dealt groups: at every slot k all eight XCDs run the same column tile
  for (int k = 0; k < tg.per_dealt; ++k) {
    int tm0, tn0;
    tile_at(tg, xcd_position(tg, 0, k), 0, tm0, tn0);
    for (int x = 1; x < kNumXcd; ++x) {
      int tm, tn;
      tile_at(tg, xcd_position(tg, x, k), 0, tm, tn);
      if (tn != tn0 || tm == tm0) return fail("dealt groups aligned", tiles_m, tiles_n, k);
    }
  }
  return 0;
}

int main() {
  if (check_spread()) return 1;
  const int cases[][5] = {
      {210, 14, 80367, 3584, 1536}, {128, 14, 49152, 3584, 2512}, {12, 14, 4608, 3584, 2512},
      {210, 14, 80367, 3584, 144},  {1, 1, 300, 128, 72},        {6, 1, 2304, 128, 10},
      {3, 1, 1000, 192, 0},         {298, 14, 114432, 3584, 1536}, {2, 2, 500, 300, 3},
      {447, 14, 5000, 3584, 1},     {396, 372, 152064, 95214, 112}, {5, 6, 1920, 1536, 7},
      {132, 14, 50688, 3584, 2512}, {210, 14, 80367, 3584, 1584},  {132, 314, 50688, 80367, 112}};
  for (auto& c : cases)
    if (check_launches(c[0], c[1], c[2], c[3], c[4])) return 1;
  std::printf("ok\n");
  return 0;
}
