"""Pins for the oracle's elastic budget scheduler (Alg. 1: phase 1 depth
extension with checkpoint gating, phase 2 width expansion)."""
import numpy as np
import pytest

import oracle
from oracle import status as st
import synth
from tests import bruteforce as bf

NONE = st.MAX_DEPTH + 1


def _exact(p):
    offs, parent, logq = p["cand_offsets"], p["parent"], p["logq"]
    N = int(offs[-1])
    S = [bf.exact_path_score(offs, parent, logq, g) for g in range(N)]
    depth = [len(bf.root_path(offs, parent, g)) for g in range(N)]
    req = [int(np.searchsorted(offs, g, side="right") - 1) for g in range(N)]
    return S, depth, req


@pytest.mark.parametrize("seed", range(30))
def test_unbounded_width_without_checkpoints_is_depth_major_order(seed):
    """W_topk at least every level's width and no checkpoint: phase 1 takes whole
    levels, so the selection is the first B finite nodes in the order (depth,
    request, S descending, index)."""
    p = synth.micro_pool(np.random.default_rng(seed), 4, 9)
    S, depth, req = _exact(p)
    N = len(S)
    order = sorted((g for g in range(N) if S[g] is not None),
                   key=lambda g: (depth[g], req[g], -S[g], g))
    for budget in sorted({0, 1, 3, N // 2, N, N + 4}):
        res = oracle.elastic_schedule(p["cand_offsets"], p["parent"], p["logq"], budget, [], [],
                                      w_topk=N + 1, w_max=N + 1)
        assert set(np.nonzero(res["selected"])[0].tolist()) == set(order[:budget]), budget
        assert res["num_selected"] == min(budget, len(order))
        assert res["status"] == 0


@pytest.mark.parametrize("seed", range(20))
def test_width_one_grows_greedy_chains_round_robin(seed):
    """W_topk = 1, no checkpoint: every request grows its greedy chain (best
    child of the last node), one depth per round, requests in order."""
    p = synth.micro_pool(np.random.default_rng(100 + seed), 5, 10)
    offs, parent = p["cand_offsets"], p["parent"]
    S, depth, req = _exact(p)
    R = len(offs) - 1
    chains = []
    for r in range(R):
        lo, hi = int(offs[r]), int(offs[r + 1])
        chain, cur = [], -1
        while True:
            kids = [g for g in range(lo, hi) if int(parent[g]) == (cur - lo if cur >= 0 else -1)
                    and S[g] is not None]
            if not kids:
                break
            cur = min(kids, key=lambda g: (-S[g], g))
            chain.append(cur)
        chains.append(chain)
    rounds = [(d, r) for d in range(1, 17) for r in range(R) if len(chains[r]) >= d]
    for budget in (0, 2, R, 2 * R + 1, len(rounds), len(rounds) + 3):
        want = {chains[r][d - 1] for d, r in rounds[:budget]}
        res = oracle.elastic_schedule(offs, parent, p["logq"], budget, [], [], w_topk=1, w_max=1)
        assert set(np.nonzero(res["selected"])[0].tolist()) == want, budget


@pytest.mark.parametrize("seed", range(20))
def test_unbounded_budget_and_width_equals_sparse_truncation(seed):
    """With budget and widths that never bind, the schedule keeps exactly the
    nodes above each request's first failed checkpoint: the sparse gate's set."""
    rng = np.random.default_rng(300 + seed)
    p = synth.micro_pool(rng, 4, 10)
    N = int(p["cand_offsets"][-1])
    sig = sorted(rng.choice(np.arange(1, 6), int(rng.integers(1, 4)), replace=False).tolist())
    lt = rng.choice([-0.25, -0.5, -0.75, -1.0, -np.inf], len(sig)).astype(np.float32)
    res = oracle.elastic_schedule(p["cand_offsets"], p["parent"], p["logq"], N + 1, sig, lt,
                                  w_topk=N + 1, w_max=N + 1)
    ref = oracle.gate_sparse(p["cand_offsets"], p["parent"], p["logq"], N + 1, sig, lt)
    assert np.array_equal(res["selected"], ref["selected"])


def test_worked_example():
    """Hand-derived.  Request 0: S = -0.25, -0.5 | -0.5, -0.75 | -1.0, -1.0 by depth;
    request 1: S = -0.5, -1.0 | -1.5, -1.25, -2.0.  Checkpoint at depth 2 with
    ln tau = -1.0, W_topk = 1, W_max = 2."""
    offs = np.array([0, 6, 11], np.int32)
    parent = np.array([-1, -1, 0, 0, 2, 3, -1, -1, 0, 1, 0], np.int32)
    logq = np.array([-0.25, -0.5, -0.25, -0.5, -0.5, -0.25,
                     -0.5, -1.0, -1.0, -0.25, -1.5], np.float32)
    run = lambda B, wmax=2: oracle.elastic_schedule(offs, parent, logq, B, [2],
                                                    np.array([-1.0], np.float32), 1, wmax)
    # depth 1: nodes 0 and 6; depth 2: request 0 passes (-0.5 > -1) and takes 2,
    # request 1's only appendable nodes (children of 6) peak at -1.5: truncated;
    # depth 3: request 0 takes 4; depth 4: nothing left.  Phase 2 widens request
    # 1's depth 1 by one node (7).
    r5 = run(5)
    assert r5["selected"].tolist() == [1, 0, 1, 0, 1, 0, 1, 1, 0, 0, 0]
    assert r5["trunc_depth"].tolist() == [NONE, 2]
    assert r5["width"][1, 1] == 2
    # budget 4 is spent in phase 1
    assert run(4)["selected"].tolist() == [1, 0, 1, 0, 1, 0, 1, 0, 0, 0, 0]
    # budget 3 runs out before request 1 is tested at depth 2: it is never truncated
    r3 = run(3)
    assert r3["selected"].tolist() == [1, 0, 1, 0, 0, 0, 1, 0, 0, 0, 0]
    assert r3["trunc_depth"].tolist() == [NONE, NONE]
    # W_max = 1: no room to widen
    assert run(5, wmax=1)["selected"].tolist() == [1, 0, 1, 0, 1, 0, 1, 0, 0, 0, 0]
    # a larger budget leaves some unspent: only 5 nodes are reachable
    r6 = run(6, wmax=3)
    assert r6["num_selected"] == 5
    # the plain top-B spends the same budget differently
    assert oracle.gate(offs, parent, logq, 5)["selected"].tolist() == \
        [1, 1, 1, 1, 0, 0, 1, 0, 0, 0, 0]


@pytest.mark.parametrize("seed", range(20))
def test_invariants(seed):
    rng = np.random.default_rng(900 + seed)
    p = synth.micro_pool(rng, 5, 14)
    offs, parent = p["cand_offsets"], p["parent"]
    S, depth, req = _exact(p)
    N = len(S)
    wt, wm = int(rng.integers(1, 4)), int(rng.integers(0, 6))
    sig = [1, 3]
    lt = np.array([-0.6, -1.6], np.float32)
    for budget in (1, N // 3, N):
        res = oracle.elastic_schedule(offs, parent, p["logq"], budget, sig, lt, wt, wm)
        sel = res["selected"].astype(bool)
        assert bf.closed(offs, parent, np.nonzero(sel)[0].tolist())
        assert res["num_selected"] <= budget
        for g in np.nonzero(sel)[0]:
            assert S[g] is not None
            assert depth[g] < res["trunc_depth"][req[g]]
        for r in range(len(offs) - 1):
            t = res["trunc_depth"][r]
            for d in range(1, 17):
                cap = max(wt, wm) if d == t - 1 else wt
                assert res["width"][r, d] <= cap
                assert res["width"][r, d] == sum(1 for g in range(N) if sel[g] and req[g] == r
                                                 and depth[g] == d)


def test_phase_two_serves_truncated_requests_in_request_order():
    """Hand-derived: requests 0 and 1 both fail the depth-2 checkpoint; the one
    unit of budget left after phase 1 widens request 0, not request 1."""
    # each request: two root children (S = -0.5, -0.75) and one grandchild (S = -2.5)
    offs = np.array([0, 3, 6], np.int32)
    parent = np.array([-1, -1, 0, -1, -1, 0], np.int32)
    logq = np.array([-0.5, -0.75, -2.0] * 2, np.float32)
    res = oracle.elastic_schedule(offs, parent, logq, 3, [2], np.array([-1.0], np.float32),
                                  w_topk=1, w_max=2)
    assert res["trunc_depth"].tolist() == [2, 2]
    assert res["selected"].tolist() == [1, 1, 0, 1, 0, 0]
    # with budget for both, both widen
    res = oracle.elastic_schedule(offs, parent, logq, 4, [2], np.array([-1.0], np.float32),
                                  w_topk=1, w_max=2)
    assert res["selected"].tolist() == [1, 1, 0, 1, 1, 0]
