"""Pins of the reference owner planner (Algorithm 1) against hand-worked plans, brute force and
the classical bound of largest-first greedy scheduling."""
import itertools

import numpy as np
import pytest

from oracle import planner as P


def test_hand_worked_plans():
    # block 0: matrices 10 and 5 and a tail of 3; block 1: one matrix of 7; two ranks
    params = [(0, 10, True), (0, 5, True), (0, 3, False), (1, 7, True)]
    # ScopeGreedy: 10 -> r0, 7 -> r1, 5 -> r1 (7 < 10), 3 -> r0 (10 < 12)
    assert P.plan(params, 2, P.SCOPE_GREEDY) == ([0, 1, 0, 1], P.SCOPE_GREEDY)
    # RoleGreedy: block 0: 10 -> r0, 5 -> r1, 3 -> r1; block 1 (loads 10, 8): 7 -> r1
    assert P.plan(params, 2, P.ROLE_GREEDY) == ([0, 1, 1, 1], P.ROLE_GREEDY)
    assert P.rank_loads(params, [0, 1, 1, 1], 2) == [10, 15]
    # CostAware: scope's max load 13 < role's 15, no cap -> scope
    assert P.plan(params, 2, P.COST_AWARE) == ([0, 1, 0, 1], P.SCOPE_GREEDY)


def test_tail_is_one_role():
    params = [(0, 4, False), (0, 4, False), (0, 6, True)]
    owner, _ = P.plan(params, 3, P.SCOPE_GREEDY)
    assert owner[0] == owner[1]            # the two non-2D tensors form one tail role of 8
    assert owner == [0, 0, 1]              # tail (8) first, then the matrix (6)
    P.validate(params, owner, 3)


def test_equal_roles_go_round_robin():
    params = [(b, 5, True) for b in range(7)]
    owner, _ = P.plan(params, 3, P.SCOPE_GREEDY)
    assert owner == [0, 1, 2, 0, 1, 2, 0]


def test_enough_ranks_one_role_each():
    rng = np.random.default_rng(60)
    params = [(int(b), int(n), True) for b, n in zip(rng.integers(0, 4, 9), rng.integers(1, 1000, 9))]
    owner, _ = P.plan(params, 12, P.SCOPE_GREEDY)
    assert len(set(owner)) == 9
    assert owner[int(np.argmax([p[1] for p in params]))] == 0


def test_single_block_role_equals_scope():
    rng = np.random.default_rng(61)
    params = [(0, int(n), bool(m)) for n, m in zip(rng.integers(1, 500, 20), rng.integers(0, 2, 20))]
    assert P.role_greedy(params, 5) == P.scope_greedy(params, 5)


def _opt_makespan(sizes, world):
    best = None
    for assign in itertools.product(range(world), repeat=len(sizes)):
        loads = [0] * world
        for s, r in zip(sizes, assign):
            loads[r] += s
        m = max(loads)
        best = m if best is None else min(best, m)
    return best


@pytest.mark.parametrize("seed", range(12))
def test_scope_greedy_within_graham_bound(seed):
    # largest-first greedy on identical machines: makespan <= (4/3 - 1/(3W)) OPT (Graham 1969)
    rng = np.random.default_rng(100 + seed)
    W = int(rng.integers(2, 4))
    k = int(rng.integers(3, 8))
    sizes = [int(x) for x in rng.integers(1, 60, k)]
    params = [(int(rng.integers(0, 3)), s, True) for s in sizes]
    owner = P.scope_greedy(params, W)
    mk = max(P.rank_loads(params, owner, W))
    opt = _opt_makespan(sizes, W)
    assert mk * 3 * W <= (4 * W - 1) * opt


def test_loads_and_gamma_invariants():
    rng = np.random.default_rng(62)
    params = [(int(b), int(n), bool(m)) for b, n, m in
              zip(rng.integers(0, 6, 60), rng.integers(1, 10000, 60), rng.integers(0, 2, 60))]
    for pol in (P.ROLE_GREEDY, P.SCOPE_GREEDY, P.COST_AWARE):
        owner, _ = P.plan(params, 8, pol)
        P.validate(params, owner, 8)
        assert sum(P.rank_loads(params, owner, 8)) == sum(p[1] for p in params)
        for g in P.block_gamma(params, owner, 8).values():
            assert 1.0 - 1e-12 <= g <= 8.0 + 1e-12
    # a block with a single role puts all of it on one rank: gamma_B = W
    owner, _ = P.plan([(0, 100, True), (1, 50, True), (1, 50, True)], 4, P.SCOPE_GREEDY)
    assert P.block_gamma([(0, 100, True), (1, 50, True), (1, 50, True)], owner, 4)[0] == 4.0


def test_cost_aware_respects_the_cap():
    params = [(0, 10, True), (0, 5, True), (0, 3, False), (1, 7, True)]
    sg = P.scope_greedy(params, 2)
    worst = max(P.block_gamma(params, sg, 2).values())
    assert P.plan(params, 2, P.COST_AWARE, cap=worst)[1] == P.SCOPE_GREEDY
    assert P.plan(params, 2, P.COST_AWARE, cap=worst * 0.99)[1] == P.ROLE_GREEDY


# ------------------------------------------------------------------ per-block layouts (Section 4.1)

def test_layouts_hand_worked():
    params = [(0, 10, True), (0, 5, True), (0, 3, False), (1, 7, True)]
    owner = [0, 1, 0, 1]                      # the ScopeGreedy plan worked above
    g, l, lens = P.layouts(params, owner, 2)
    # block 0 canonical: [0, 10) [10, 15) [15, 18); block 1: [0, 7)
    assert g == [0, 10, 15, 0]
    # rank 0 holds the matrix of 10 (first index 0) then the tail (first index 2); rank 1 the 5
    assert l == [0, 0, 10, 0]
    assert lens == [[13, 5], [0, 7]]
    P.validate_layouts(params, owner, 2, g, l, lens)


def test_layouts_tail_packed_before_a_later_matrix():
    # non-2D tensors at indices 0 and 2 around a matrix: the tail (first index 0) comes first in its
    # owner's buffer and its two tensors are packed next to each other
    params = [(0, 4, False), (0, 6, True), (0, 2, False), (0, 8, True)]
    owner, _ = P.plan(params, 2, P.SCOPE_GREEDY)
    assert owner == [1, 1, 1, 0]              # 8 -> r0; matrix 6 (before the tail of 6 on ties) -> r1; tail -> r1
    g, l, lens = P.layouts(params, owner, 2)
    assert g == [0, 4, 10, 12]
    assert l == [0, 6, 4, 0]
    assert lens == [[8, 12]]
    P.validate_layouts(params, owner, 2, g, l, lens)


def test_layouts_of_random_plans_are_valid():
    rng = np.random.default_rng(70)
    for _ in range(200):
        n = int(rng.integers(0, 25))
        params = [(int(rng.integers(0, 5)), int(rng.integers(0, 50)), bool(rng.integers(0, 2))) for _ in range(n)]
        world = int(rng.integers(1, 7))
        for pol in (P.ROLE_GREEDY, P.SCOPE_GREEDY):
            owner, _ = P.plan(params, world, pol)
            g, l, lens = P.layouts(params, owner, world)
            P.validate_layouts(params, owner, world, g, l, lens)
            # rank r's buffers over all blocks hold exactly its load
            assert [sum(lens[b][r] for b in range(len(lens))) for r in range(world)] == P.rank_loads(params, owner, world)


def test_layout_validation_rejects_broken_layouts():
    params = [(0, 10, True), (0, 5, True), (0, 3, False), (0, 2, False), (1, 7, True)]
    owner = [0, 1, 0, 0, 1]
    g, l, lens = P.layouts(params, owner, 2)
    P.validate_layouts(params, owner, 2, g, l, lens)
    bad = list(l)
    bad[1] += 1                               # a gap in rank 1's buffer
    with pytest.raises(ValueError):
        P.validate_layouts(params, owner, 2, g, bad, lens)
    bad = list(l)
    bad[2], bad[3] = l[3], l[2]               # the tail out of parameter order
    with pytest.raises(ValueError):
        P.validate_layouts(params, owner, 2, g, bad, lens)
    with pytest.raises(ValueError):
        P.validate_layouts(params, owner, 2, g, l, [[13, 5], [0, 8]])
    with pytest.raises(ValueError):
        P.layouts(params, [0, 1, 0, 1, 1], 2)  # the block's tail split across ranks


def test_layouts_with_empty_tensors():
    # an empty tail tensor after a matrix in parameter order, but packed with the tail before it
    params = [(0, 3, False), (0, 4, True), (0, 0, False), (0, 0, True)]
    owner = [0, 0, 0, 0]
    g, l, lens = P.layouts(params, owner, 1)
    assert g == [0, 3, 7, 7] and l == [0, 3, 3, 7] and lens == [[7]]
    P.validate_layouts(params, owner, 1, g, l, lens)
