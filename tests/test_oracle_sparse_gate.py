"""Pins for the oracle's sparse checkpoint gating (eq. 6, eq. 7; Alg. 1 phase 1
truncation) followed by the global top-B of eq. 4."""
import itertools
import math

import numpy as np
import pytest

import oracle
from oracle import status as st
import synth
from tests import bruteforce as bf


def _exact(offs, parent, logq):
    N = int(offs[-1])
    S = [bf.exact_path_score(offs, parent, logq, g) for g in range(N)]
    depth = [len(bf.root_path(offs, parent, g)) for g in range(N)]
    req = [int(np.searchsorted(offs, g, side="right") - 1) for g in range(N)]
    return S, depth, req


def _eligible(offs, parent, logq, sig_depth, log_tau):
    """Quantifier form of the truncation, on exact path sums: a node survives iff
    for every checkpoint (d, ln tau) with d <= its depth, some node of its
    request at depth d has a path score strictly above ln tau."""
    S, depth, req = _exact(offs, parent, logq)
    N = len(S)
    ok = []
    for g in range(N):
        good = True
        for d, lt in zip(sig_depth, log_tau):
            if d > depth[g]:
                continue
            witness = any(req[m] == req[g] and depth[m] == d and S[m] is not None
                          and S[m] > lt for m in range(N))
            good = good and witness
        ok.append(good)
    return ok, S


def _brute_sparse(offs, parent, logq, budget, sig_depth, log_tau):
    """Best ancestor-closed subset (sum exp S) among surviving finite nodes,
    lexicographically first among ties."""
    ok, S = _eligible(offs, parent, logq, sig_depth, log_tau)
    cands = [g for g in range(len(S)) if ok[g] and S[g] is not None]
    m = min(budget, len(cands))
    best, best_val = (), None
    for comb in itertools.combinations(cands, m):
        if not bf.closed(offs, parent, comb):
            continue
        val = math.fsum(math.exp(float(S[g])) for g in comb)
        if best_val is None or val > best_val + 1e-12 * abs(best_val) or (
                abs(val - best_val) <= 1e-12 * abs(best_val) and comb < best):
            best, best_val = comb, val
    return set(best)


@pytest.mark.parametrize("seed", range(40))
def test_sparse_gate_matches_exhaustive_search(seed):
    rng = np.random.default_rng(500 + seed)
    p = synth.micro_pool(rng, 3, 6)
    offs, parent, logq = p["cand_offsets"], p["parent"], p["logq"]
    N = int(offs[-1])
    nsig = int(rng.integers(1, 4))
    sig = sorted(rng.choice(np.arange(1, 5), nsig, replace=False).tolist())
    # thresholds on the same dyadic grid as the scores: equality (a failed strict
    # test) happens often
    lt = [float(x) for x in rng.choice([-0.25, -0.5, -0.75, -1.0, -1.5, 0.0, -np.inf], nsig)]
    for budget in sorted({0, 1, 2, N // 2, N, N + 2}):
        res = oracle.gate_sparse(offs, parent, logq, budget, sig, np.array(lt, np.float32))
        want = _brute_sparse(offs, parent, logq, budget, sig, lt)
        got = set(np.nonzero(res["selected"])[0].tolist())
        assert got == want, (seed, budget, sig, lt)
        assert res["num_selected"] == len(want)
        assert res["status"] == 0


@pytest.mark.parametrize("seed", range(10))
def test_no_checkpoint_or_zero_threshold_is_plain_top_b(seed):
    """D_sig empty, or tau = 0 (ln tau = -inf) at every depth where a finite
    node exists: nothing is truncated and the plain top-B results."""
    b = synth.micro_pool(np.random.default_rng(seed), 5, 12, p_neg_inf=0.0)
    offs, parent, logq = b["cand_offsets"], b["parent"], b["logq"]
    N = int(offs[-1])
    for budget in (0, 3, N // 2, N):
        ref = oracle.gate(offs, parent, logq, budget)
        a = oracle.gate_sparse(offs, parent, logq, budget, [], np.zeros(0, np.float32))
        z = oracle.gate_sparse(offs, parent, logq, budget, [1, 2, 3],
                               np.full(3, -np.inf, np.float32))
        assert np.array_equal(a["selected"], ref["selected"])
        assert np.array_equal(z["selected"], ref["selected"])
        assert np.array_equal(a["path_score"], ref["path_score"])


def test_tau_one_truncates_at_the_first_checkpoint():
    """tau = 1 (ln tau = 0): max S > 0 is impossible (log q <= 0), so every
    request stops before the smallest checkpoint depth."""
    b = synth.micro_pool(np.random.default_rng(3), 6, 14, p_neg_inf=0.0)
    offs, parent, logq = b["cand_offsets"], b["parent"], b["logq"]
    N = int(offs[-1])
    depth = np.array([len(bf.root_path(offs, parent, g)) for g in range(N)])
    res = oracle.gate_sparse(offs, parent, logq, N, [4, 2], np.zeros(2, np.float32))
    assert np.array_equal(res["selected"].astype(bool), depth < 2)
    assert np.all(res["trunc_depth"][np.diff(offs) > 0] == 2)


def test_worked_example_budget_moves_to_the_confident_request():
    """Hand-derived: request 1 fails the depth-2 checkpoint, its depth-2 budget
    goes to request 0's next node."""
    offs = np.array([0, 4, 8], np.int32)
    parent = np.array([-1, -1, 0, 0, -1, -1, 0, 2], np.int32)
    logq = np.array([-0.25, -1.0, -0.5, -2.0, -0.5, -0.75, -0.5, -0.25], np.float32)
    # S = [-0.25, -1, -0.75, -2.25, -0.5, -0.75, -1.0, -1.25]
    plain = oracle.gate(offs, parent, logq, 6)
    assert plain["selected"].tolist() == [1, 1, 1, 0, 1, 1, 1, 0]
    sp = oracle.gate_sparse(offs, parent, logq, 6, [2], np.array([-0.8], np.float32))
    assert sp["trunc_depth"].tolist() == [st.MAX_DEPTH + 1, 2]
    assert sp["selected"].tolist() == [1, 1, 1, 1, 1, 1, 0, 0]
    # the checkpoint test is strict: ln tau equal to the depth-2 maximum fails
    eq = oracle.gate_sparse(offs, parent, logq, 6, [2], np.array([-0.75], np.float32))
    assert eq["trunc_depth"].tolist() == [2, 2]
    assert eq["selected"].tolist() == [1, 1, 0, 0, 1, 1, 0, 0]
    # a depth-1 checkpoint that only request 0 passes
    d1 = oracle.gate_sparse(offs, parent, logq, 3, [1], np.array([-0.4], np.float32))
    assert d1["trunc_depth"].tolist() == [st.MAX_DEPTH + 1, 1]
    assert d1["selected"].tolist() == [1, 1, 1, 0, 0, 0, 0, 0]


def test_layer_confidence_is_the_depth_maximum():
    """eq. 6 before the exp: the per-(request, depth) maximum of S."""
    b = synth.micro_pool(np.random.default_rng(9), 4, 10)
    offs, parent, logq = b["cand_offsets"], b["parent"], b["logq"]
    S, depth, req = _exact(offs, parent, logq)
    res = oracle.gate_sparse(offs, parent, logq, 5, [1], np.full(1, -np.inf, np.float32))
    for r in range(len(offs) - 1):
        for d in range(1, st.MAX_DEPTH + 1):
            vals = [float(S[g]) for g in range(len(S)) if req[g] == r and depth[g] == d
                    and S[g] is not None]
            want = max(vals) if vals else -np.inf
            assert float(res["layer_max"][r, d]) == want, (r, d)


def test_fixed_threshold_on_a_chain_stops_where_the_score_crosses():
    """Fixed tau at every depth on single chains: S falls along the chain, so
    the first failed depth is the first node at or below ln tau."""
    logq = np.array([-0.25, -0.5, -0.25, -1.0, -0.5], np.float32)
    # S = -0.25, -0.75, -1.0, -2.0, -2.5
    offs = np.array([0, 5], np.int32)
    parent = np.array([-1, 0, 1, 2, 3], np.int32)
    for lt, t in [(-0.1, 1), (-0.5, 2), (-1.0, 3), (-1.5, 4), (-2.25, 5), (-3.0, 6)]:  # depth 6 is empty: fails
        res = oracle.gate_sparse(offs, parent, logq, 5, list(range(1, 17)),
                                 np.full(16, lt, np.float32))
        assert res["trunc_depth"].tolist() == [t], lt
        assert res["selected"].tolist() == [1 if d < t else 0 for d in range(1, 6)]
