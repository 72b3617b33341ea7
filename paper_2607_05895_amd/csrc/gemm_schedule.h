// Tile schedules of the grouped NS products (host side; plain C++ with no HIP dependency, so that
// the CPU tests can build and check it on its own).
#pragma once

#include <stdint.h>

#include <algorithm>
#include <cstdint>
#include <cstring>
#include <vector>

namespace mfsdp {

// One output tile of a grouped NS product: problem (matrix) index, block coordinates (in tiles of
// the launch: 256 x 256, or 128 x 128) and, for a problem whose contraction is split, the K range ks
// of the tile; e < 0 marks an idle slot. The bf16 NS kernels run a persistent grid of kGemmXcds x S
// workgroups (S = kGemmSlots on 256 x 256 tiles, one workgroup per CU; twice that on 128 x 128
// tiles); workgroup b serves XCD b % kGemmXcds, slot b / kGemmXcds, and takes tile
// sched[g * S + slot] of every group g = xcd, xcd + kGemmXcds, ...
struct TileRef {
  int32_t e;
  int16_t bi, bj;
  int16_t ks;
  int16_t unused;
};
constexpr int kGemmXcds = 8;    // MI355X: 8 XCDs (workgroups are dealt to them round robin)
constexpr int kGemmSlots = 32;  // CUs per XCD = tiles per group
constexpr int kGroupRows = 4;   // a group covers 4 block rows x 8 block columns of one matrix

// Per-problem tile grid of one NS product (256 x 256 tiles on the bf16 path).
struct TileGrid {
  int tm, tn;
  bool sym;
};

// Tile schedule of one product for the persistent bf16 kernel. Tiles are put in locality order
// (bands of group_rows block rows, within a band column by column, upper triangle only for
// symmetric products) and cut into groups of `slots` tiles, so that the workgroups of one XCD
// run the tiles of a group together and share its operand blocks in L2. Groups are then dealt to
// the XCDs longest first, each to the XCD with the least work so far (a group's cost is the
// largest K among its tiles: its tiles run side by side). Group g of the result runs on XCD
// g % kGemmXcds; XCDs with fewer groups get empty ones (every slot e = -1).
// splits (optional, per problem): the number of K ranges each tile of the problem is cut into; the
// ranges of one tile are listed together and each costs cost / splits. fill (<= slots, default
// slots): tiles per group; a group's remaining slots stay idle, which spreads a launch with few
// tiles over more XCDs.
inline std::vector<TileRef> build_schedule(const std::vector<int>& order, const std::vector<TileGrid>& grids,
                                           const std::vector<int64_t>& cost,
                                           const std::vector<int>* splits = nullptr,
                                           int slots = kGemmSlots, int group_rows = kGroupRows,
                                           int fill = 0) {
  if (fill <= 0 || fill > slots) fill = slots;
  auto nks = [&](int e) { return splits ? (*splits)[e] : 1; };
  std::vector<TileRef> flat;
  for (int e : order) {
    const TileGrid& g = grids[e];
    for (int r0 = 0; r0 < g.tm; r0 += group_rows) {
      const int r1 = std::min(g.tm, r0 + group_rows);
      for (int c = g.sym ? r0 : 0; c < g.tn; ++c)
        for (int r = r0; r < r1; ++r)
          if (!g.sym || r <= c)
            for (int ks = 0; ks < nks(e); ++ks) flat.push_back(TileRef{e, int16_t(r), int16_t(c), int16_t(ks), 0});
    }
  }
  if (fill < slots) {  // spread: fill tiles, then slots - fill idle ones, per group
    std::vector<TileRef> spread;
    for (size_t i = 0; i < flat.size(); ++i) {
      spread.push_back(flat[i]);
      if ((i + 1) % size_t(fill) == 0 || i + 1 == flat.size())
        while (spread.size() % size_t(slots)) spread.push_back(TileRef{-1, 0, 0, 0, 0});
    }
    flat.swap(spread);
  }
  while (flat.size() % size_t(slots)) flat.push_back(TileRef{-1, 0, 0, 0, 0});
  const size_t ng = flat.size() / size_t(slots);
  std::vector<int64_t> gcost(ng, 0);
  for (size_t g = 0; g < ng; ++g)
    for (int s = 0; s < slots; ++s) {
      const TileRef& t = flat[g * size_t(slots) + size_t(s)];
      if (t.e >= 0) gcost[g] = std::max(gcost[g], cost[t.e] / nks(t.e));
    }
  std::vector<size_t> by(ng);
  for (size_t g = 0; g < ng; ++g) by[g] = g;
  std::stable_sort(by.begin(), by.end(), [&](size_t x, size_t y) { return gcost[x] > gcost[y]; });
  std::vector<std::vector<size_t>> lists(kGemmXcds);
  int64_t load[kGemmXcds] = {};
  for (size_t g : by) {
    int best = 0;
    for (int x = 1; x < kGemmXcds; ++x)
      if (load[x] < load[best]) best = x;
    lists[best].push_back(g);
    load[best] += gcost[g];
  }
  size_t rounds = 0;
  for (const auto& l : lists) rounds = std::max(rounds, l.size());
  std::vector<TileRef> s(rounds * kGemmXcds * size_t(slots), TileRef{-1, 0, 0, 0, 0});
  for (int x = 0; x < kGemmXcds; ++x)
    for (size_t i = 0; i < lists[x].size(); ++i)
      std::memcpy(&s[(i * kGemmXcds + size_t(x)) * size_t(slots)], &flat[lists[x][i] * size_t(slots)],
                  size_t(slots) * sizeof(TileRef));
  return s;
}

// K splits of a Gram product launch (upper tiles tiles[e] of contraction length K[e] per problem)
// with fewer tiles than the persistent grid has workgroups (slots: the grid's workgroups). A tile's time is set by its K, so a
// few long-K tiles (say those of a 768 x 3072 matrix among 768 x 768 ones) would alone set the
// launch's length while most of the chip waits. Each problem gets the largest f <= kSplitMax that
// divides K / 32 and keeps K / f at least at a target: first the larger of kSplitMinK and the
// launch's work per workgroup, then the longest K range any problem is left with (so that no tile
// is cut shorter than the launch needs). f = 1 everywhere when the launch fills the grid. The split
// problems' partial tiles (tiles x f each) are held to max_parts: while over, the problem with the
// most ranges (the most tiles among equals, then the first) drops to its next smaller count.
constexpr int64_t kSplitMinK = 512;
constexpr int kSplitMax = 8;
inline std::vector<int> gram_splits(const std::vector<int64_t>& tiles, const std::vector<int64_t>& K,
                                    int64_t max_parts = INT64_MAX,
                                    int64_t slots = int64_t(kGemmXcds) * kGemmSlots) {
  const size_t n = tiles.size();
  std::vector<int> f(n, 1);
  int64_t T = 0, W = 0;
  for (size_t e = 0; e < n; ++e) {
    T += tiles[e];
    W += tiles[e] * K[e];
  }
  if (n == 0 || T >= slots) return f;
  auto fit = [](int64_t k, int64_t target) {
    int best = 1;
    for (int c = 2; c <= kSplitMax; ++c)
      if ((k / 32) % c == 0 && k / c >= target) best = c;
    return best;
  };
  const int64_t kt = std::max(kSplitMinK, W / slots);
  int64_t kcrit = 0;
  for (size_t e = 0; e < n; ++e) kcrit = std::max(kcrit, K[e] / fit(K[e], kt));
  for (size_t e = 0; e < n; ++e) f[e] = fit(K[e], kcrit);
  auto parts = [&] {
    int64_t p = 0;
    for (size_t e = 0; e < n; ++e)
      if (f[e] > 1) p += tiles[e] * f[e];
    return p;
  };
  while (parts() > max_parts) {
    size_t w = 0;
    for (size_t e = 1; e < n; ++e)
      if (f[e] > f[w] || (f[e] == f[w] && tiles[e] > tiles[w])) w = e;
    int c = f[w] - 1;
    while (c > 1 && (K[w] / 32) % c != 0) --c;
    f[w] = c;
  }
  return f;
}

}  // namespace mfsdp
