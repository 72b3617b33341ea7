"""Reference owner planner (test infrastructure only: only tests/, __graft_entry__.smoke() and
bench.py's cpu_baseline use this package; the library has its own C++ planner).

Paper passages followed:
* Section 4.1 ("MatrixShard: representing ownership"): each block is converted into roles, one per
  2D matrix and one packed tail of the block's non-2D tensors; the greedy load is the owner-resident
  numel.
* Algorithm 1 ("Balance-aware owner planning"): RoleGreedy assigns each block's roles, largest
  first, to the currently lightest ranks and carries the loads into the next block; ScopeGreedy pools
  the roles of all blocks and assigns them largest first to the lightest ranks; CostAware keeps the
  scope plan only if it improves balance within the workspace caps, else uses RoleGreedy; every
  parameter ends up as one contiguous segment on one rank.
* Section 4.2 ("Owner-segment communication collectives", bandwidth model): for block B with P_B
  elements over shard span W, gamma_B = max_r O_{B,r} / (P_B / W).

Readings (the paper gives no tie rules and no cap definition):
* roles of equal size keep their order: by block, then matrices in parameter order, then the tail;
  the lightest rank is the lowest-numbered among equally loaded ranks;
* RoleGreedy visits blocks in increasing block index;
* "balance improves" means a strictly smaller maximum rank load; the workspace cap bounds gamma_B
  of every block (cap <= 0: no cap).
"""
from __future__ import annotations

from typing import Dict, List, Sequence, Tuple

ROLE_GREEDY, SCOPE_GREEDY, COST_AWARE = 0, 1, 2


def build_roles(params: Sequence[Tuple[int, int, bool]]):
    """params: (block, numel, is_matrix) per parameter. Returns the roles as
    (block, numel, order_key, [parameter indices]) with order_key = (block, kind, first index)
    where kind 0 = matrix, 1 = tail."""
    roles = []
    tails: Dict[int, List[int]] = {}
    for i, (blk, numel, is_matrix) in enumerate(params):
        if numel < 0:
            raise ValueError("numel must be >= 0")
        if is_matrix:
            roles.append((blk, numel, (blk, 0, i), [i]))
        else:
            tails.setdefault(blk, []).append(i)
    for blk, idx in tails.items():
        roles.append((blk, sum(params[i][1] for i in idx), (blk, 1, idx[0]), idx))
    return roles


def _assign(roles, loads: List[int], owner: List[int]) -> None:
    # largest role first; equal sizes keep their order key; the lightest rank, lowest index on ties
    for blk, numel, key, idx in sorted(roles, key=lambda r: (-r[1], r[2])):
        r = min(range(len(loads)), key=lambda k: (loads[k], k))
        loads[r] += numel
        for i in idx:
            owner[i] = r


def role_greedy(params, world: int) -> List[int]:
    roles = build_roles(params)
    owner = [-1] * len(params)
    loads = [0] * world
    for blk in sorted({r[0] for r in roles}):
        _assign([r for r in roles if r[0] == blk], loads, owner)
    return owner


def scope_greedy(params, world: int) -> List[int]:
    owner = [-1] * len(params)
    _assign(build_roles(params), [0] * world, owner)
    return owner


def rank_loads(params, owner: Sequence[int], world: int) -> List[int]:
    loads = [0] * world
    for (blk, numel, _), r in zip(params, owner):
        loads[r] += numel
    return loads


def block_gamma(params, owner: Sequence[int], world: int) -> Dict[int, float]:
    """gamma_B = max_r O_{B,r} / (P_B / W) for every block with P_B > 0."""
    per: Dict[int, List[int]] = {}
    for (blk, numel, _), r in zip(params, owner):
        per.setdefault(blk, [0] * world)[r] += numel
    out = {}
    for blk, o in per.items():
        total = sum(o)
        if total > 0:
            out[blk] = max(o) / (total / world)
    return out


def cost_aware(params, world: int, cap: float) -> Tuple[List[int], int]:
    """Returns (owner, policy actually used)."""
    rg = role_greedy(params, world)
    sg = scope_greedy(params, world)
    better = max(rank_loads(params, sg, world)) < max(rank_loads(params, rg, world))
    within = cap <= 0 or all(g <= cap for g in block_gamma(params, sg, world).values())
    return (sg, SCOPE_GREEDY) if (better and within) else (rg, ROLE_GREEDY)


def plan(params, world: int, policy: int, cap: float = 0.0) -> Tuple[List[int], int]:
    if world < 1:
        raise ValueError("world must be >= 1")
    if policy == ROLE_GREEDY:
        return role_greedy(params, world), ROLE_GREEDY
    if policy == SCOPE_GREEDY:
        return scope_greedy(params, world), SCOPE_GREEDY
    if policy == COST_AWARE:
        return cost_aware(params, world, cap)
    raise ValueError("unknown policy")


def validate(params, owner: Sequence[int], world: int) -> None:
    """One owner per parameter, in range; a block's non-2D tensors share one owner (its tail)."""
    tails: Dict[int, int] = {}
    for (blk, numel, is_matrix), r in zip(params, owner):
        if not 0 <= r < world:
            raise ValueError("owner out of range")
        if not is_matrix:
            if tails.setdefault(blk, r) != r:
                raise ValueError("a block's tail is split across ranks")
