"""The library's C++ owner planner (Algorithm 1 with the gamma_B model of Section 4.2) against the
pinned Python oracle: identical owners, rank loads, per-block gamma_B and chosen policy on random
instances with many ties, on the paper's decoder shapes, and on the degenerate cases. Host only."""
import math

import numpy as np
import pytest

import synth
from oracle import planner as P
from paper_2607_05895_amd import native

POLICIES = (P.ROLE_GREEDY, P.SCOPE_GREEDY, P.COST_AWARE)


def _oracle(params, world, policy, cap):
    owner, used = P.plan(params, world, policy, cap)
    loads = P.rank_loads(params, owner, world)
    nblocks = 1 + max((b for b, _, _ in params), default=-1)
    g = P.block_gamma(params, owner, world)
    gam = [g.get(b, 0.0) for b in range(nblocks)]
    return owner, loads, gam, used


def _check(params, world, policy, cap=0.0):
    got = native.mfsdp_plan_owners(params, world, policy, cap)
    exp = _oracle(params, world, policy, cap)
    assert got[0] == exp[0], "owners"
    assert got[1] == exp[1], "rank loads"
    assert got[2] == exp[2], "gamma_B (bitwise: same evaluation order in double)"
    assert got[3] == exp[3], "policy used"
    P.validate(params, got[0], world)
    # the per-block layouts of the plan, bit for bit, and valid
    lay = native.mfsdp_plan_layouts(params, world, got[0])
    assert lay == tuple(P.layouts(params, got[0], world)), "layouts"
    P.validate_layouts(params, got[0], world, *lay)
    return got


@pytest.mark.parametrize("seed", range(60))
def test_random_instances_match_oracle(seed):
    rng = np.random.Generator(np.random.PCG64(seed))
    params = synth.random_plan_params(rng, blocks=int(rng.integers(1, 9)),
                                      max_numel=int(rng.choice([3, 50, 4096])))
    world = int(rng.integers(1, 12))
    for policy in POLICIES:
        _check(params, world, policy)
    # a cap between the two plans' gamma values exercises both CostAware outcomes
    sg = _oracle(params, world, P.SCOPE_GREEDY, 0.0)[2]
    for cap in (0.0, -1.0, 1.0, max(sg, default=0.0), 0.5 * (1.0 + max(sg, default=1.0)), 1e9):
        _check(params, world, P.COST_AWARE, cap)


@pytest.mark.parametrize("layers,world", [(16, 8), (32, 16), (64, 32), (128, 64)])
def test_paper_sweep_shapes_match_oracle(layers, world):
    # latency/memory sweep model: hidden 4096, intermediate 16384, layers grow with the span
    params = [p.tuple() for p in synth.decoder_plan_params(layers)]
    for policy in POLICIES:
        _check(params, world, policy)


def test_convergence_model_matches_oracle():
    params = [p.tuple() for p in synth.decoder_plan_params(12, 768, 3072, vocab=50257, norm="layer")]
    for world in (1, 8, 64):
        for policy in POLICIES:
            _check(params, world, policy)


def test_cost_aware_choice_both_ways():
    # role plan {10,5,3 | 7} on 2 ranks: loads 10/15; scope plan 13/12 -> scope balances better
    params = [(0, 10, True), (0, 5, True), (0, 3, False), (1, 7, True)]
    owner, loads, gam, used = _check(params, 2, P.COST_AWARE, 0.0)
    assert used == P.SCOPE_GREEDY and max(loads) == 13
    # block 1 (one matrix of 7) has gamma 2 under any plan; a cap below it rejects the scope plan
    assert gam[1] == 2.0
    assert _check(params, 2, P.COST_AWARE, 1.9)[3] == P.ROLE_GREEDY
    assert _check(params, 2, P.COST_AWARE, 2.0)[3] == P.SCOPE_GREEDY


def test_degenerate_cases():
    assert native.mfsdp_plan_owners([], 4, P.COST_AWARE) == ([], [0, 0, 0, 0], [], P.ROLE_GREEDY)
    params = [(0, 8, True), (0, 8, True), (2, 0, False)]
    o, loads, gam, used = _check(params, 1, P.SCOPE_GREEDY)
    assert o == [0, 0, 0] and loads == [16] and gam == [1.0, 0.0, 0.0]
    # more ranks than roles: every role alone, ranks beyond them idle
    o, loads, gam, _ = _check(params, 16, P.ROLE_GREEDY)
    assert o[:2] == [0, 1] and sum(loads) == 16 and gam[0] == 8.0
    # all-zero sizes: every plan has max load 0, CostAware keeps RoleGreedy
    _check([(0, 0, True), (1, 0, False), (1, 0, True)], 3, P.COST_AWARE)
    # large numel (beyond 32 bits)
    big = [(0, 1 << 40, True), (0, (1 << 40) + 1, True), (1, 3, False)]
    assert _check(big, 2, P.SCOPE_GREEDY)[1] == [(1 << 40) + 1, (1 << 40) + 3]


def test_invalid_arguments_rejected():
    with pytest.raises(native.MfsdpError, match="world"):
        native.mfsdp_plan_owners([(0, 1, True)], 0, P.ROLE_GREEDY)
    with pytest.raises(native.MfsdpError, match="policy"):
        native.mfsdp_plan_owners([(0, 1, True)], 2, 3)
    with pytest.raises(native.MfsdpError, match="NaN"):
        native.mfsdp_plan_owners([(0, 1, True)], 2, P.COST_AWARE, math.nan)
    with pytest.raises(native.MfsdpError, match="numel"):
        native.mfsdp_plan_owners([(0, -1, True)], 2, P.ROLE_GREEDY)
    with pytest.raises(native.MfsdpError, match="block"):
        native.mfsdp_plan_owners([(-1, 1, True)], 2, P.ROLE_GREEDY)
    # NULL owner with count > 0 through the raw symbol
    import ctypes
    arr = (native.PlanParam * 1)(native.PlanParam(0, 1, 1))
    st = native.lib().mfsdp_plan_owners(arr, 1, 2, 0, 0.0, None, None, None, None)
    assert st == native.E_INVALID


def test_layouts_hand_worked_and_rejections():
    params = [(0, 4, False), (0, 6, True), (0, 2, False), (0, 8, True)]
    assert native.mfsdp_plan_layouts(params, 2, [1, 1, 1, 0]) == ([0, 4, 10, 12], [0, 6, 4, 0], [[8, 12]])
    assert native.mfsdp_plan_layouts([], 3, []) == ([], [], [])
    with pytest.raises(native.MfsdpError, match="tail is split"):
        native.mfsdp_plan_layouts(params, 2, [1, 1, 0, 0])
    with pytest.raises(native.MfsdpError, match="owner out of range"):
        native.mfsdp_plan_layouts(params, 2, [1, 1, 1, 2])
    with pytest.raises(native.MfsdpError, match="world"):
        native.mfsdp_plan_layouts(params, 0, [0, 0, 0, 0])
    # sparse block indices and empty tensors: blocks without parameters get all-zero rows
    params = [(3, 5, True), (3, 0, False), (1, 2, False), (1, 0, True)]
    lay = native.mfsdp_plan_layouts(params, 2, [1, 0, 0, 1])
    assert lay == tuple(P.layouts(params, [1, 0, 0, 1], 2))
    assert lay[2][0] == [0, 0] and lay[2][2] == [0, 0]
