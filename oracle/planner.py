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

Layouts (Section 4.1, "MatrixShard": a rank-indexed placement of each flattened parameter interval;
Algorithm 1's last step: one layout per block, validated for one contiguous local segment per
parameter). Readings (the paper does not fix the packing order):
* a block's canonical axis is its parameters' flattened elements concatenated in parameter order;
* a rank's local buffer for a block holds the roles of that block it owns, ordered by each role's
  first parameter index; a matrix role is the whole matrix, the tail role the block's non-2D
  tensors packed in parameter order (one whole segment on the tail owner);
* a parameter's local segment on any other rank is empty.
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


def layouts(params, owner: Sequence[int], world: int):
    """Per-block MatrixShard layouts of a plan. Returns (global_offset, local_offset, lengths):
    global_offset[i] and local_offset[i] are parameter i's offsets on its block's canonical axis and
    in its owner's local buffer of that block; lengths[b][r] is rank r's local buffer length in
    block b (blocks 0 .. max block)."""
    validate(params, owner, world)
    nblocks = 1 + max((p[0] for p in params), default=-1)
    lengths = [[0] * world for _ in range(nblocks)]
    canon = [0] * nblocks
    global_offset = [0] * len(params)
    local_offset = [0] * len(params)
    # canonical axis: parameter order within each block
    for i, (blk, numel, _) in enumerate(params):
        global_offset[i] = canon[blk]
        canon[blk] += numel
    # local buffers: roles in the order of their first parameter index
    roles = sorted(build_roles(params), key=lambda r: r[3][0])
    for blk, numel, _, idx in roles:
        r = owner[idx[0]]
        pos = lengths[blk][r]
        for i in idx:                 # one parameter (a matrix), or the tail in parameter order
            local_offset[i] = pos
            pos += params[i][1]
        lengths[blk][r] = pos
    return global_offset, local_offset, lengths


def validate_layouts(params, owner: Sequence[int], world: int, global_offset, local_offset, lengths) -> None:
    """Algorithm 1's last step: every parameter is one contiguous segment of its numel on its owner
    (empty elsewhere); every rank's segments tile its local buffer of each block exactly; a block's
    tail is one contiguous segment in parameter order; the local buffers of a block hold its whole
    canonical axis, whose intervals tile [0, P_B) in parameter order."""
    validate(params, owner, world)
    nblocks = 1 + max((p[0] for p in params), default=-1)
    if len(lengths) != nblocks or any(len(row) != world for row in lengths):
        raise ValueError("one row of rank lengths per block")
    canon = [0] * nblocks
    segs = {}
    for i, (blk, numel, _) in enumerate(params):
        if global_offset[i] != canon[blk]:
            raise ValueError(f"parameter {i}: canonical interval out of order")
        canon[blk] += numel
        segs.setdefault((blk, owner[i]), []).append((local_offset[i], numel, i))
    for b in range(nblocks):
        if sum(lengths[b]) != canon[b]:
            raise ValueError(f"block {b}: local buffers hold {sum(lengths[b])} of {canon[b]} elements")
        for r in range(world):
            pos = 0
            # at one offset, empty segments first (an empty tail tensor may share its offset with
            # the role that follows the tail)
            for off, numel, i in sorted(segs.get((b, r), []), key=lambda t: (t[0], t[1] > 0, t[2])):
                if off != pos:
                    raise ValueError(f"block {b} rank {r}: parameter {i} at {off}, expected {pos}")
                pos += numel
            if pos != lengths[b][r]:
                raise ValueError(f"block {b} rank {r}: segments cover {pos} of {lengths[b][r]}")
    tails = {}
    for i, (blk, numel, is_matrix) in enumerate(params):
        if not is_matrix:
            tails.setdefault(blk, []).append(i)
    for blk, idx in tails.items():
        for a, b in zip(idx, idx[1:]):
            if local_offset[b] != local_offset[a] + params[a][1]:
                raise ValueError(f"block {blk}: tail not packed in parameter order")
