// Owner planner (Section 4.1, Algorithm 1 "Balance-aware owner planning") and the per-block
// bandwidth ratio gamma_B of the owner-segment collectives (Section 4.2). Host code only.
//
// Roles: every 2D matrix of a block is one role; the block's non-2D tensors form one packed tail
// role. The load of a rank is the numel it owns. RoleGreedy visits the blocks in increasing index
// and gives each block's roles, largest first, to the currently lightest rank, carrying the loads
// from block to block; ScopeGreedy does the same over the roles of all blocks at once; CostAware
// keeps the scope plan only when its largest rank load is strictly smaller than RoleGreedy's and
// every block's gamma_B stays within the cap. Ties: roles of equal size keep their order (block,
// matrices before the tail, parameter index); the lightest rank is the lowest-numbered of equally
// loaded ranks. gamma_B = max_r O_{B,r} / (P_B / W), evaluated in that order in double.
#include <stdint.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <functional>
#include <queue>
#include <string>
#include <unordered_map>
#include <utility>
#include <vector>

#include "../../include/mfsdp.h"

namespace mfsdp {
int set_last_error(int status, const std::string& msg);  // defined with the other entry points
}

namespace {

struct Role {
  int64_t numel;
  int32_t block;
  int32_t kind;   // 0 matrix, 1 tail
  int64_t first;  // first parameter index
};

bool role_before(const Role& x, const Role& y) {
  if (x.numel != y.numel) return x.numel > y.numel;
  if (x.block != y.block) return x.block < y.block;
  if (x.kind != y.kind) return x.kind < y.kind;
  return x.first < y.first;
}

// Roles of the parameters and the role of every parameter.
void build_roles(const mfsdp_plan_param* params, int64_t count, std::vector<Role>& roles,
                 std::vector<int64_t>& role_of) {
  roles.clear();
  role_of.assign(size_t(count), -1);
  std::unordered_map<int32_t, int64_t> tail;  // block -> role index
  for (int64_t i = 0; i < count; ++i) {
    const mfsdp_plan_param& p = params[i];
    if (p.is_matrix) {
      role_of[i] = int64_t(roles.size());
      roles.push_back(Role{p.numel, p.block, 0, i});
    } else {
      auto it = tail.find(p.block);
      if (it == tail.end()) {
        it = tail.emplace(p.block, int64_t(roles.size())).first;
        roles.push_back(Role{0, p.block, 1, i});
      }
      roles[size_t(it->second)].numel += p.numel;
      role_of[i] = it->second;
    }
  }
}

using Heap = std::priority_queue<std::pair<int64_t, int32_t>, std::vector<std::pair<int64_t, int32_t>>,
                                 std::greater<std::pair<int64_t, int32_t>>>;

// Largest role first to the lightest rank; `order` lists role indices.
void assign(const std::vector<Role>& roles, std::vector<int64_t>& order, Heap& heap,
            std::vector<int32_t>& role_owner) {
  std::stable_sort(order.begin(), order.end(),
                   [&](int64_t a, int64_t b) { return role_before(roles[size_t(a)], roles[size_t(b)]); });
  for (int64_t ri : order) {
    auto top = heap.top();
    heap.pop();
    role_owner[size_t(ri)] = top.second;
    heap.push({top.first + roles[size_t(ri)].numel, top.second});
  }
}

Heap fresh_heap(int32_t world) {
  Heap h;
  for (int32_t r = 0; r < world; ++r) h.push({0, r});
  return h;
}

std::vector<int32_t> role_greedy(const std::vector<Role>& roles, int32_t world) {
  std::vector<int32_t> owner(roles.size(), -1);
  std::vector<int64_t> idx(roles.size());
  for (size_t i = 0; i < roles.size(); ++i) idx[i] = int64_t(i);
  std::stable_sort(idx.begin(), idx.end(),
                   [&](int64_t a, int64_t b) { return roles[size_t(a)].block < roles[size_t(b)].block; });
  Heap heap = fresh_heap(world);
  for (size_t s = 0; s < idx.size();) {
    size_t e = s;
    while (e < idx.size() && roles[size_t(idx[e])].block == roles[size_t(idx[s])].block) ++e;
    std::vector<int64_t> blk(idx.begin() + long(s), idx.begin() + long(e));
    assign(roles, blk, heap, owner);
    s = e;
  }
  return owner;
}

std::vector<int32_t> scope_greedy(const std::vector<Role>& roles, int32_t world) {
  std::vector<int32_t> owner(roles.size(), -1);
  std::vector<int64_t> idx(roles.size());
  for (size_t i = 0; i < roles.size(); ++i) idx[i] = int64_t(i);
  Heap heap = fresh_heap(world);
  assign(roles, idx, heap, owner);
  return owner;
}

int64_t max_load(const std::vector<Role>& roles, const std::vector<int32_t>& owner, int32_t world) {
  std::vector<int64_t> load(size_t(world), 0);
  for (size_t i = 0; i < roles.size(); ++i) load[size_t(owner[i])] += roles[i].numel;
  return *std::max_element(load.begin(), load.end());
}

// gamma_B of every block 0 .. nblocks-1 (0 for blocks without elements)
std::vector<double> gammas(const std::vector<Role>& roles, const std::vector<int32_t>& owner,
                           int32_t world, int32_t nblocks) {
  std::unordered_map<int64_t, int64_t> o;  // block * world + rank -> owned numel
  std::vector<int64_t> total(size_t(nblocks), 0), mx(size_t(nblocks), 0);
  for (size_t i = 0; i < roles.size(); ++i) {
    const int64_t key = int64_t(roles[i].block) * world + owner[i];
    const int64_t v = (o[key] += roles[i].numel);
    total[size_t(roles[i].block)] += roles[i].numel;
    mx[size_t(roles[i].block)] = std::max(mx[size_t(roles[i].block)], v);
  }
  std::vector<double> g(size_t(nblocks), 0.0);
  for (int32_t b = 0; b < nblocks; ++b)
    if (total[size_t(b)] > 0) g[size_t(b)] = double(mx[size_t(b)]) / (double(total[size_t(b)]) / double(world));
  return g;
}

}  // namespace

extern "C" int mfsdp_plan_owners(const mfsdp_plan_param* params, int64_t count, int32_t world,
                                 int32_t policy, double gamma_cap, int32_t* owner,
                                 int64_t* rank_load, double* block_gamma, int32_t* policy_used) {
  using mfsdp::set_last_error;
  if (count < 0) return set_last_error(MFSDP_E_INVALID, "count must be >= 0");
  if (count > 0 && (!params || !owner)) return set_last_error(MFSDP_E_INVALID, "params and owner must be non-NULL");
  if (world < 1 || world > (1 << 16)) return set_last_error(MFSDP_E_INVALID, "world must be in [1, 65536]");
  if (policy < MFSDP_PLAN_ROLE_GREEDY || policy > MFSDP_PLAN_COST_AWARE)
    return set_last_error(MFSDP_E_INVALID, "unknown policy");
  if (std::isnan(gamma_cap)) return set_last_error(MFSDP_E_INVALID, "gamma_cap is NaN");
  int32_t nblocks = 0;
  for (int64_t i = 0; i < count; ++i) {
    if (params[i].block < 0 || params[i].numel < 0 || (params[i].is_matrix != 0 && params[i].is_matrix != 1))
      return set_last_error(MFSDP_E_INVALID, "param " + std::to_string(i) + ": block and numel must be >= 0, is_matrix 0 or 1");
    nblocks = std::max(nblocks, params[i].block + 1);
  }
  std::vector<Role> roles;
  std::vector<int64_t> role_of;
  build_roles(params, count, roles, role_of);
  std::vector<int32_t> ro;
  int32_t used = policy;
  if (policy == MFSDP_PLAN_ROLE_GREEDY) {
    ro = role_greedy(roles, world);
  } else if (policy == MFSDP_PLAN_SCOPE_GREEDY) {
    ro = scope_greedy(roles, world);
  } else {
    std::vector<int32_t> rg = role_greedy(roles, world), sg = scope_greedy(roles, world);
    bool take = roles.empty() ? false : max_load(roles, sg, world) < max_load(roles, rg, world);
    if (take && gamma_cap > 0.0) {
      for (double g : gammas(roles, sg, world, nblocks))
        if (g > gamma_cap) take = false;
    }
    ro = take ? sg : rg;
    used = take ? MFSDP_PLAN_SCOPE_GREEDY : MFSDP_PLAN_ROLE_GREEDY;
  }
  for (int64_t i = 0; i < count; ++i) owner[i] = ro[size_t(role_of[size_t(i)])];
  if (rank_load) {
    for (int32_t r = 0; r < world; ++r) rank_load[r] = 0;
    for (size_t i = 0; i < roles.size(); ++i) rank_load[ro[i]] += roles[i].numel;
  }
  if (block_gamma) {
    const std::vector<double> g = gammas(roles, ro, world, nblocks);
    for (int32_t b = 0; b < nblocks; ++b) block_gamma[b] = g[size_t(b)];
  }
  if (policy_used) *policy_used = used;
  return MFSDP_OK;
}

// Per-block MatrixShard layouts of a plan (Section 4.1; the last step of Algorithm 1). A block's
// canonical axis concatenates its parameters in parameter order; a rank's local buffer for a block
// holds the roles of that block it owns in the order of each role's first parameter index (a
// matrix whole, the tail's tensors packed in parameter order). The emitted layout is then
// validated: per rank and block the segments tile the local buffer exactly, the tail is packed in
// parameter order, and the block's local buffers hold its whole canonical axis.
extern "C" int mfsdp_plan_layouts(const mfsdp_plan_param* params, int64_t count, int32_t world,
                                  const int32_t* owner, int64_t* global_offset, int64_t* local_offset,
                                  int64_t* block_rank_len) {
  using mfsdp::set_last_error;
  if (count < 0) return set_last_error(MFSDP_E_INVALID, "count must be >= 0");
  if (count > 0 && (!params || !owner || !global_offset || !local_offset))
    return set_last_error(MFSDP_E_INVALID, "params, owner and the offset arrays must be non-NULL");
  if (world < 1 || world > (1 << 16)) return set_last_error(MFSDP_E_INVALID, "world must be in [1, 65536]");
  int32_t nblocks = 0;
  std::unordered_map<int32_t, int32_t> tail_owner;
  std::unordered_map<int32_t, int64_t> tail_numel;
  for (int64_t i = 0; i < count; ++i) {
    const mfsdp_plan_param& p = params[i];
    if (p.block < 0 || p.numel < 0 || (p.is_matrix != 0 && p.is_matrix != 1))
      return set_last_error(MFSDP_E_INVALID, "param " + std::to_string(i) + ": block and numel must be >= 0, is_matrix 0 or 1");
    if (owner[i] < 0 || owner[i] >= world)
      return set_last_error(MFSDP_E_INVALID, "param " + std::to_string(i) + ": owner out of range");
    if (!p.is_matrix) {
      auto it = tail_owner.emplace(p.block, owner[i]).first;
      if (it->second != owner[i])
        return set_last_error(MFSDP_E_INVALID, "block " + std::to_string(p.block) + ": its tail is split across ranks");
      tail_numel[p.block] += p.numel;
    }
    nblocks = std::max(nblocks, p.block + 1);
  }
  std::unordered_map<int32_t, int64_t> canon;                 // block -> canonical length so far
  std::unordered_map<int64_t, int64_t> len;                   // block * world + rank -> local length
  std::unordered_map<int32_t, int64_t> tail_pos;              // block -> next tail offset
  for (int64_t i = 0; i < count; ++i) {
    const mfsdp_plan_param& p = params[i];
    global_offset[i] = canon[p.block];
    canon[p.block] += p.numel;
    const int64_t key = int64_t(p.block) * world + owner[i];
    if (p.is_matrix) {
      local_offset[i] = len[key];
      len[key] += p.numel;
    } else {
      auto it = tail_pos.find(p.block);
      if (it == tail_pos.end()) {  // the tail role starts at its first tensor: reserve all of it
        it = tail_pos.emplace(p.block, len[key]).first;
        len[key] += tail_numel[p.block];
      }
      local_offset[i] = it->second;
      it->second += p.numel;
    }
  }
  // validation: segments tile every local buffer, the tail is packed in parameter order, and the
  // local buffers of a block add up to its canonical axis
  std::unordered_map<int64_t, std::vector<std::pair<std::pair<int64_t, int>, int64_t>>> segs;
  for (int64_t i = 0; i < count; ++i)
    segs[int64_t(params[i].block) * world + owner[i]].push_back({{local_offset[i], params[i].numel > 0 ? 1 : 0}, i});
  for (auto& kv : segs) {
    auto& v = kv.second;
    std::sort(v.begin(), v.end());
    int64_t pos = 0;
    for (const auto& sg : v) {
      if (sg.first.first != pos)
        return set_last_error(MFSDP_E_INVALID, "layout: parameter " + std::to_string(sg.second) + " leaves a gap or overlaps");
      pos += params[sg.second].numel;
    }
    if (pos != len[kv.first]) return set_last_error(MFSDP_E_INVALID, "layout: local buffer not covered");
  }
  std::unordered_map<int32_t, int64_t> last_tail;  // block -> index of the previous tail tensor
  std::unordered_map<int32_t, int64_t> local_sum;
  for (const auto& kv : len) local_sum[int32_t(kv.first / world)] += kv.second;
  for (int64_t i = 0; i < count; ++i) {
    if (params[i].is_matrix) continue;
    auto it = last_tail.find(params[i].block);
    if (it != last_tail.end() && local_offset[i] != local_offset[it->second] + params[it->second].numel)
      return set_last_error(MFSDP_E_INVALID, "layout: tail of block " + std::to_string(params[i].block) + " not packed");
    last_tail[params[i].block] = i;
  }
  for (const auto& kv : canon)
    if (local_sum[kv.first] != kv.second) return set_last_error(MFSDP_E_INVALID, "layout: block not covered");
  if (block_rank_len) {
    for (int64_t b = 0; b < nblocks; ++b)
      for (int32_t r = 0; r < world; ++r) {
        auto it = len.find(b * world + r);
        block_rank_len[b * world + r] = it == len.end() ? 0 : it->second;
      }
  }
  return MFSDP_OK;
}
