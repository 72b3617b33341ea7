// CPU check of the NS GEMM tile schedules (gemm_schedule.h): every tile of every problem exactly
// once (upper triangle only for symmetric products; every K range of a split problem's tile once),
// whole rounds of XCD groups, every group's tiles on one XCD, the deal's balance (the busiest XCD
// within one group of the mean), and determinism; random launches plus the owner shares' own
// launches, on the 256 x 256 grid (one workgroup per CU) and the 128 x 128 one (two); the Gram
// launches' K splits (gram_splits) on hand-worked cases. Exit code 0 on
// success; every failure prints what it found.
#include <cstdio>
#include <map>
#include <random>
#include <tuple>

#include "gemm_schedule.h"

using namespace mfsdp;

static int g_fail = 0;
#define CHECK(c, ...)                                  \
  do {                                                 \
    if (!(c)) {                                        \
      ++g_fail;                                        \
      std::printf("FAIL %s:%d: ", __FILE__, __LINE__); \
      std::printf(__VA_ARGS__);                        \
      std::printf("\n");                               \
    }                                                  \
  } while (0)

static void check_launch(const std::vector<TileGrid>& grids, const std::vector<int64_t>& cost,
                         const std::vector<int>* splits = nullptr, int slots = kGemmSlots,
                         int group_rows = kGroupRows, int fill = 0) {
  std::vector<int> pos(grids.size());
  for (size_t k = 0; k < pos.size(); ++k) pos[k] = int(k);
  auto nks = [&](int e) { return splits ? (*splits)[e] : 1; };
  const std::vector<TileRef> s = build_schedule(pos, grids, cost, splits, slots, group_rows, fill);
  const std::vector<TileRef> s2 = build_schedule(pos, grids, cost, splits, slots, group_rows, fill);
  CHECK(s.size() == s2.size() && std::memcmp(s.data(), s2.data(), s.size() * sizeof(TileRef)) == 0,
        "not deterministic");
  const size_t round = size_t(kGemmXcds) * size_t(slots);
  CHECK(s.size() % round == 0, "%zu slots: not whole rounds", s.size());
  std::map<std::tuple<int, int, int, int>, int> seen;
  int64_t load[kGemmXcds] = {};
  int64_t ntiles = 0, total = 0, gmax = 0;
  for (size_t e = 0; e < grids.size(); ++e) {
    const TileGrid& g = grids[e];
    ntiles += (g.sym ? int64_t(g.tm) * (g.tm + 1) / 2 : int64_t(g.tm) * g.tn) * nks(int(e));
  }
  for (size_t g = 0; g < s.size() / size_t(slots); ++g) {
    int64_t gc = 0;
    for (int sl = 0; sl < slots; ++sl) {
      const TileRef& t = s[g * size_t(slots) + size_t(sl)];
      if (t.e < 0) continue;
      CHECK(fill <= 0 || sl < fill, "tile in slot %d of a group filled to %d", sl, fill);
      CHECK(t.e < int(grids.size()), "problem %d", t.e);
      const TileGrid& gr = grids[t.e];
      CHECK(t.bi >= 0 && t.bi < gr.tm && t.bj >= 0 && t.bj < gr.tn && (!gr.sym || t.bi <= t.bj),
            "tile (%d, %d) outside problem %d", t.bi, t.bj, t.e);
      CHECK(t.ks >= 0 && t.ks < nks(t.e), "K range %d of problem %d (%d ranges)", t.ks, t.e, nks(t.e));
      seen[std::make_tuple(int(t.e), int(t.bi), int(t.bj), int(t.ks))] += 1;
      gc = std::max(gc, cost[t.e] / nks(t.e));
    }
    load[g % kGemmXcds] += gc;   // group g runs on XCD g % kGemmXcds
    total += gc;
    gmax = std::max(gmax, gc);
  }
  CHECK(int64_t(seen.size()) == ntiles, "%zu of %lld tiles scheduled", seen.size(), (long long)ntiles);
  for (const auto& kv : seen) CHECK(kv.second == 1, "a tile scheduled %d times", kv.second);
  int64_t busiest = 0;
  for (int x = 0; x < kGemmXcds; ++x) busiest = std::max(busiest, load[x]);
  // greedy longest-first deal: the busiest XCD exceeds the mean by at most one group
  CHECK(busiest * kGemmXcds <= total + int64_t(kGemmXcds) * gmax, "unbalanced deal: %lld of %lld",
        (long long)busiest, (long long)total);
}

static void share(const char* name, const std::vector<std::pair<int, int>>& shapes) {
  // the three products of one NS step, problems in the launch's order (longest K first)
  for (int ph = 0; ph < 3; ++ph) {
    std::vector<std::pair<int, int>> ord = shapes;  // (r_pad, s_pad)
    std::stable_sort(ord.begin(), ord.end(), [&](auto a, auto b) {
      return (ph == 0 ? a.second : a.first) > (ph == 0 ? b.second : b.first);
    });
    std::vector<TileGrid> grids;
    std::vector<int64_t> cost;
    for (auto [r, s] : ord) {
      const int tr = r / 256, ts = s / 256;
      grids.push_back(ph == 2 ? TileGrid{tr, ts, false} : TileGrid{tr, tr, true});
      cost.push_back(ph == 0 ? s : r);
    }
    check_launch(grids, cost);
  }
  std::printf("%s: ok\n", name);
}

int main() {
  std::mt19937 rng(12345);
  for (int it = 0; it < 400; ++it) {
    const int np = 1 + rng() % 8;
    std::vector<TileGrid> grids;
    std::vector<int64_t> cost;
    for (int e = 0; e < np; ++e) {
      const int tr = 1 + rng() % 24, ts = tr + rng() % 60;
      grids.push_back(rng() % 3 == 2 ? TileGrid{tr, ts, false} : TileGrid{tr, tr, true});
      cost.push_back(256 * (1 + int64_t(rng() % 64)));
    }
    std::stable_sort(cost.begin(), cost.end(), std::greater<int64_t>());
    check_launch(grids, cost);
    check_launch(grids, cost, nullptr, 2 * kGemmSlots, 2 * kGroupRows);
    check_launch(grids, cost, nullptr, 2 * kGemmSlots, 2 * kGroupRows, kGemmSlots);
  }
  std::printf("random launches: ok\n");
  share("gpt2_small_share", {{768, 768}, {768, 768}, {768, 768}, {768, 768}, {768, 768}, {768, 768},
                             {768, 768}, {768, 768}, {768, 3072}, {768, 3072}, {768, 3072}, {768, 3072}});
  std::vector<std::pair<int, int>> l8, l70;
  for (int l = 0; l < 4; ++l)
    for (auto sh : {std::make_pair(4096, 4096), std::make_pair(1024, 4096), std::make_pair(1024, 4096),
                    std::make_pair(4096, 4096), std::make_pair(4096, 14336), std::make_pair(4096, 14336),
                    std::make_pair(4096, 14336)})
      l8.push_back(sh);
  share("llama3_8b_share", l8);
  for (auto sh : {std::make_pair(8192, 8192), std::make_pair(1024, 8192), std::make_pair(1024, 8192),
                  std::make_pair(8192, 8192), std::make_pair(8192, 28672), std::make_pair(8192, 28672),
                  std::make_pair(8192, 28672), std::make_pair(8192, 28672), std::make_pair(8192, 28672)})
    l70.push_back(sh);
  share("llama3_70b_share", l70);
  // K splits of the Gram launch (upper tiles, K): the GPT-2-small share's 768 x 3072 matrices cut in
  // 4 ranges of 768, the K of its 768 x 768 ones; one 768 x 3072 matrix alone in 6 ranges of 512
  // (96 K blocks of 32 = 6 x 16); a launch that fills the grid, and a uniform one whose work per
  // workgroup exceeds half its K, not split
  {
    std::vector<int64_t> tl, kl;
    for (int i = 0; i < 4; ++i) { tl.push_back(6); kl.push_back(3072); }
    for (int i = 0; i < 8; ++i) { tl.push_back(6); kl.push_back(768); }
    const std::vector<int> f = gram_splits(tl, kl);
    for (int i = 0; i < 12; ++i) CHECK(f[i] == (i < 4 ? 4 : 1), "gpt2 share: problem %d split %d", i, f[i]);
    std::vector<TileGrid> grids(12, TileGrid{3, 3, true});
    check_launch(grids, kl, &f);
    CHECK(gram_splits({6}, {3072})[0] == 6, "one 768 x 3072 matrix: %d", gram_splits({6}, {3072})[0]);
    CHECK(gram_splits({300}, {4096})[0] == 1, "a full launch was split");
    CHECK(gram_splits({200, 20}, {3072, 3072})[0] == 1, "a uniform launch was split");
    const std::vector<int> g2 = gram_splits({10, 10}, {8192, 256});
    CHECK(g2[0] == 8 && g2[1] == 1, "8192 / 256: %d %d", g2[0], g2[1]);
    std::vector<TileGrid> gg{TileGrid{4, 4, true}, TileGrid{4, 4, true}};
    check_launch(gg, {8192, 256}, &g2);
    // the partial-tile budget: one 2048 x 2048 matrix (36 tiles, 4 ranges uncapped) drops to 2
    // ranges under 100 partial tiles and to none under 48; the GPT-2 share's 96 fit 140
    CHECK(gram_splits({36}, {2048})[0] == 4, "2048 x 2048 uncapped: %d", gram_splits({36}, {2048})[0]);
    CHECK(gram_splits({36}, {2048}, 100)[0] == 2, "2048 x 2048 capped at 100: %d", gram_splits({36}, {2048}, 100)[0]);
    CHECK(gram_splits({36}, {2048}, 48)[0] == 1, "2048 x 2048 capped at 48: %d", gram_splits({36}, {2048}, 48)[0]);
    CHECK(gram_splits(tl, kl, 140) == f, "GPT-2 share under a 140-tile budget");
    const std::vector<int> g3 = gram_splits(tl, kl, 60);
    int64_t p3 = 0;
    for (int i = 0; i < 12; ++i) p3 += g3[i] > 1 ? tl[i] * g3[i] : 0;
    CHECK(p3 <= 60, "GPT-2 share under a 60-tile budget: %lld partial tiles", (long long)p3);
    // the same share's Gram launch on 128 x 128 tiles (21 upper tiles per matrix) and the grid of
    // two workgroups per CU: the 768 x 3072 matrices again in 4 ranges (504 tiles for 512 slots)
    const int64_t small = int64_t(kGemmXcds) * 2 * kGemmSlots;
    std::vector<int64_t> t128(12, 21);
    const std::vector<int> f128 = gram_splits(t128, kl, INT64_MAX, small);
    for (int i = 0; i < 12; ++i) CHECK(f128[i] == (i < 4 ? 4 : 1), "gpt2 share, 128: problem %d split %d", i, f128[i]);
    std::vector<TileGrid> g128(12, TileGrid{6, 6, true});
    check_launch(g128, kl, &f128, 2 * kGemmSlots, 2 * kGroupRows);
    // its square launch (252 tiles) spread to one tile per CU: 8 groups of at most 32, one per XCD
    {
      std::vector<int> pos(12);
      for (int i = 0; i < 12; ++i) pos[i] = i;
      const std::vector<int64_t> k768(12, 768);
      const std::vector<TileRef> sq = build_schedule(pos, g128, k768, nullptr, 2 * kGemmSlots, 2 * kGroupRows, kGemmSlots);
      CHECK(sq.size() == size_t(kGemmXcds) * 2 * kGemmSlots, "square spread: %zu slots", sq.size());
      check_launch(g128, k768, nullptr, 2 * kGemmSlots, 2 * kGroupRows, kGemmSlots);
    }
    CHECK(gram_splits({528}, {4096}, INT64_MAX, small)[0] == 1, "a full 128 x 128 launch was split");
  }
  std::printf("gram splits: ok\n");
  if (g_fail) {
    std::printf("%d failures\n", g_fail);
    return 1;
  }
  std::printf("schedule check ok\n");
  return 0;
}
