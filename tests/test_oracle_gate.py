"""Pins for the oracle gate: path scores (eq. 5) and the budgeted selection (eq. 4)."""
import json
import math
import os

import numpy as np
import pytest

import oracle
from oracle import status as st
import synth
from tests import bruteforce as bf

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _pool(seed, R=3, max_nodes=6):
    return synth.micro_pool(np.random.default_rng(seed), R, max_nodes)


@pytest.mark.parametrize("seed", range(60))
def test_gate_matches_exhaustive_search(seed):
    """Top-B by (S desc, index asc) == the closed subset maximising sum exp(S)
    (Theorem 2 / Proposition 1 exchange argument), ties -> smallest indices."""
    p = _pool(seed)
    offs, parent, logq = p["cand_offsets"], p["parent"], p["logq"]
    N = int(offs[-1])
    for budget in sorted({0, 1, 2, 3, N // 2, N, N + 3}):
        res = oracle.gate(offs, parent, logq, budget)
        want, S_exact = bf.brute_gate(offs, parent, logq, budget)
        got = set(np.nonzero(res["selected"])[0].tolist())
        assert got == want, (seed, budget)
        assert res["num_selected"] == len(want)
        assert res["status"] == 0
        # path scores: the dyadic inputs make the float32 fold exact
        for g in range(N):
            e = S_exact[g]
            if e is None:
                assert res["path_score"][g] == -np.inf
            else:
                assert float(res["path_score"][g]) == float(e)


def test_all_equal_logq_selects_breadth_first():
    """Equal log q: S = depth * log q, so the budget fills depth 1 first, then depth 2..."""
    rng = np.random.default_rng(7)
    p = synth.micro_pool(rng, 4, 12, logq_set=np.array([-0.5], np.float32), p_neg_inf=0.0)
    offs, parent = p["cand_offsets"], p["parent"]
    N = int(offs[-1])
    depth = np.array([len(bf.root_path(offs, parent, g)) for g in range(N)])
    bfs = sorted(range(N), key=lambda g: (depth[g], g))
    for budget in range(N + 1):
        res = oracle.gate(offs, parent, p["logq"], budget)
        assert set(np.nonzero(res["selected"])[0]) == set(bfs[:budget])


def test_budget_extremes_and_chain():
    p = _pool(3, R=4, max_nodes=8)
    offs, parent, logq = p["cand_offsets"], p["parent"], p["logq"]
    N = int(offs[-1])
    finite = np.array([bf.exact_path_score(offs, parent, logq, g) is not None for g in range(N)])
    assert oracle.gate(offs, parent, logq, 0)["num_selected"] == 0
    res = oracle.gate(offs, parent, logq, 10 * N)
    assert np.array_equal(res["selected"].astype(bool), finite)
    # one chain with log q = 0, everything else -inf: the selection is that chain
    offs1 = np.array([0, 6], np.int32)
    parent1 = np.array([-1, 0, -1, 1, 3, 2], np.int32)
    logq1 = np.array([0, 0, -np.inf, 0, 0, -np.inf], np.float32)
    res = oracle.gate(offs1, parent1, logq1, 4)
    assert res["selected"].tolist() == [1, 1, 0, 1, 1, 0]


def test_fold_order_golden():
    """Hand-derived values: the score is folded root -> leaf (eq. 5 recursion)."""
    with open(os.path.join(GOLDEN, "gate_fold_order.json")) as f:
        cases = json.load(f)["cases"]
    for c in cases:
        offs = np.array(c["cand_offsets"], np.int32)
        parent = np.array(c["parent"], np.int32)
        logq = np.array([float.fromhex(x) for x in c["logq_hex"]], np.float32)
        res = oracle.gate(offs, parent, logq, c["budget"])
        got = [float(x).hex() for x in res["path_score"]]
        assert got == c["path_score_hex"], c["name"]
        assert res["selected"].tolist() == c["selected"], c["name"]


def test_status_rules():
    offs = np.array([0, 4], np.int32)
    # NaN -> -inf (bit 0), positive -> 0 (bit 1), parent out of range -> -1 (bit 2)
    parent = np.array([-1, 0, 5, 0], np.int32)
    logq = np.array([-1.0, np.nan, 0.5, -2.0], np.float32)
    res = oracle.gate(offs, parent, logq, 4)
    assert res["status"] == st.NAN_LOGQ | st.POS_LOGQ | st.BAD_PARENT
    assert res["path_score"].tolist() == [-1.0, -np.inf, 0.0, -3.0]
    assert res["selected"].tolist() == [1, 0, 1, 1]
    # depth above 16 -> -inf (bit 3)
    n = 18
    offs = np.array([0, n], np.int32)
    parent = np.arange(-1, n - 1, dtype=np.int32)
    logq = np.full(n, -0.25, np.float32)
    res = oracle.gate(offs, parent, logq, n)
    assert res["status"] == st.TOO_DEEP
    assert res["num_selected"] == 16
    assert np.all(np.isinf(res["path_score"][16:]))


@pytest.mark.parametrize("name", ["tiny", "l8b"])
def test_gate_invariants_on_presets(name):
    b = synth.make_batch(name, 0, attention=False)
    cfg = b["cfg"]
    res = oracle.gate(b["cand_offsets"], b["parent"], b["logq"], cfg.budget)
    S, sel = res["path_score"], res["selected"].astype(bool)
    assert res["status"] == 0
    assert res["num_selected"] == min(cfg.budget, int(np.isfinite(S).sum()))
    # every selected key beats every unselected finite key
    idx = np.arange(len(S))
    worst_sel = max(zip(-S[sel], idx[sel]))
    fin_un = (~sel) & np.isfinite(S)
    if fin_un.any():
        best_un = min(zip(-S[fin_un], idx[fin_un]))
        assert worst_sel < best_un
    # root-to-leaf float32 fold agrees with the exact path sum to within depth ulps
    offs, parent, logq = b["cand_offsets"], b["parent"], b["logq"]
    for g in np.random.default_rng(0).choice(len(S), 50, replace=False):
        e = bf.exact_path_score(offs, parent, logq, int(g))
        assert abs(float(S[g]) - float(e)) <= cfg.depth * abs(float(e)) * 2.0 ** -23


@pytest.mark.parametrize("offs", [[2, 5, 9], [0, 6, 4, 9], [0, 4, 8]])
def test_malformed_csr_scores_and_selects_nothing(offs):
    """Boundary convention: a CSR that does not start at 0, end at N or rise is refused."""
    N = 9
    parent = np.array([-1, 0, 1, -1, 3, -1, 5, 6, -1], np.int32)
    logq = np.full(N, -0.5, np.float32)
    g = oracle.gate(np.array(offs, np.int32), parent, logq, 4)
    assert g["status"] == oracle.status.BAD_OFFSETS
    assert np.all(np.isneginf(g["path_score"]))
    assert g["num_selected"] == 0 and not g["selected"].any()
    assert oracle.gate(np.array([0, 3, 9], np.int32), parent, logq, 4)["num_selected"] == 4
