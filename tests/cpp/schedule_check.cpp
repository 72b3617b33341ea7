// CPU check of the NS GEMM tile schedules (gemm_schedule.h): every tile of every problem exactly
// once (upper triangle only for symmetric products), whole rounds of XCD groups, every group's
// tiles on one XCD, the deal's balance (the busiest XCD within one group of the mean), and
// determinism; random launches plus the owner shares' own launches. Exit code 0 on success; every
// failure prints what it found.
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

static void check_launch(const std::vector<TileGrid>& grids, const std::vector<int64_t>& cost) {
  std::vector<int> pos(grids.size());
  for (size_t k = 0; k < pos.size(); ++k) pos[k] = int(k);
  const std::vector<TileRef> s = build_schedule(pos, grids, cost);
  const std::vector<TileRef> s2 = build_schedule(pos, grids, cost);
  CHECK(s.size() == s2.size() && std::memcmp(s.data(), s2.data(), s.size() * sizeof(TileRef)) == 0,
        "not deterministic");
  const size_t round = size_t(kGemmXcds) * kGemmSlots;
  CHECK(s.size() % round == 0, "%zu slots: not whole rounds", s.size());
  std::map<std::tuple<int, int, int>, int> seen;
  int64_t load[kGemmXcds] = {};
  int64_t ntiles = 0, total = 0, gmax = 0;
  for (const TileGrid& g : grids) ntiles += g.sym ? int64_t(g.tm) * (g.tm + 1) / 2 : int64_t(g.tm) * g.tn;
  for (size_t g = 0; g < s.size() / kGemmSlots; ++g) {
    int64_t gc = 0;
    for (int sl = 0; sl < kGemmSlots; ++sl) {
      const TileRef& t = s[g * kGemmSlots + sl];
      if (t.e < 0) continue;
      CHECK(t.e < int(grids.size()), "problem %d", t.e);
      const TileGrid& gr = grids[t.e];
      CHECK(t.bi >= 0 && t.bi < gr.tm && t.bj >= 0 && t.bj < gr.tn && (!gr.sym || t.bi <= t.bj),
            "tile (%d, %d) outside problem %d", t.bi, t.bj, t.e);
      seen[std::make_tuple(int(t.e), int(t.bi), int(t.bj))] += 1;
      gc = std::max(gc, cost[t.e]);
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
  if (g_fail) {
    std::printf("%d failures\n", g_fail);
    return 1;
  }
  std::printf("schedule check ok\n");
  return 0;
}
