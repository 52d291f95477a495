"""GPU parity of sparse checkpoint gating (eq. 6-7, Alg. 1 phase 1 truncation,
then the global top-B): echo_gate_sparse against oracle.gate_sparse, bit for bit
(path scores, selection, count, truncation depths, status)."""
import sys

import numpy as np
import pytest

import oracle
import synth
from oracle import status as st
from tests import gpu_common as gc

pytestmark = pytest.mark.gpu

# checkpoint tables of the paper's appendix (first draft depth read as depth 1)
PAPER_TAU = {"l8b": {1: 0.2, 5: 0.35, 8: 0.5}, "q235b": {1: 0.15, 3: 0.3, 5: 0.5}}


@pytest.fixture(autouse=True)
def _need_gpu():
    gc.require_gpu()


def _log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def run_sparse(offs, parent, logq, budget, sig, log_tau, with_trunc=True):
    import torch
    import paper_2604_09603_amd as pkg
    from paper_2604_09603_amd.step import _aligned_workspace
    d = "cuda:0"
    R, N = len(offs) - 1, int(offs[-1])
    t = lambda a, dt: torch.from_numpy(np.ascontiguousarray(a).astype(dt)).to(d)
    path = torch.full((max(N, 1),), float("nan"), dtype=torch.float32, device=d)
    sel = torch.full((max(N, 1),), 7, dtype=torch.uint8, device=d)
    nsel = torch.full((1,), -1, dtype=torch.int32, device=d)
    trunc = torch.full((R,), -5, dtype=torch.int32, device=d) if with_trunc else None
    status = torch.zeros(1, dtype=torch.int32, device=d)
    ws = _aligned_workspace(pkg.gate_workspace_size(R, N, budget), d)
    ws.fill_(0xAB)  # the workspace's contents on entry must not matter
    pkg.echo_gate_sparse(t(offs, np.int32), t(parent, np.int32), t(logq, np.float32), R, N,
                         budget, sig, log_tau, path, sel, nsel, ws, trunc_depth=trunc,
                         status=status)
    torch.cuda.synchronize()
    return dict(path_score=path.cpu().numpy()[:N], selected=sel.cpu().numpy()[:N],
                num_selected=int(nsel.item()), status=int(status.item()),
                trunc_depth=None if trunc is None else trunc.cpu().numpy())


def check(offs, parent, logq, budget, sig, log_tau):
    lt = np.asarray(log_tau, np.float32)
    ref = oracle.gate_sparse(offs, parent, logq, budget, list(sig), lt)
    got = run_sparse(offs, parent, logq, budget, list(sig), lt.tolist())
    assert np.array_equal(got["path_score"].view(np.uint32), ref["path_score"].view(np.uint32))
    assert np.array_equal(got["selected"], ref["selected"]), "selection differs"
    assert got["num_selected"] == ref["num_selected"]
    assert np.array_equal(got["trunc_depth"], ref["trunc_depth"]), "truncation depths differ"
    assert got["status"] == ref["status"]
    return ref


def _median_table(b, depths):
    S, depth, _ = oracle.path_scores(b["cand_offsets"], b["parent"], b["logq"])
    from oracle.gate import layer_max_scores
    lm = layer_max_scores(b["cand_offsets"], S, depth)
    return [float(np.float32(np.median(lm[:, d]))) for d in depths]


@pytest.mark.parametrize("name,seed", [(n, s) for n in ["tiny", "l8b", "l70b", "q235b", "long"]
                                       for s in (0, 1)])
def test_presets_with_median_thresholds(name, seed):
    """Checkpoints at depths 1, 3, 5 with ln tau at the median layer maximum:
    about half the requests stop at each checkpoint."""
    b = synth.make_batch(name, seed, attention=False)
    sig = [1, 3, 5]
    lt = _median_table(b, sig)
    _log(f"[sparse] {name} seed={seed} ln tau={lt}")
    ref = check(b["cand_offsets"], b["parent"], b["logq"], b["cfg"].budget, sig, lt)
    t = ref["trunc_depth"]
    assert (t < st.MAX_DEPTH + 1).any() and (t == st.MAX_DEPTH + 1).any() or name == "tiny"


@pytest.mark.parametrize("name", sorted(PAPER_TAU))
def test_presets_with_paper_thresholds(name):
    b = synth.make_batch(name, 2, attention=False)
    tab = PAPER_TAU[name]
    sig = sorted(tab)
    lt = [float(np.log(np.float32(tab[d]))) for d in sig]
    _log(f"[sparse] {name} paper table {tab}")
    check(b["cand_offsets"], b["parent"], b["logq"], b["cfg"].budget, sig, lt)


@pytest.mark.parametrize("seed", range(16))
def test_micro_pools_with_ties(seed):
    rng = np.random.default_rng(700 + seed)
    p = synth.micro_pool(rng, int(rng.integers(1, 7)), int(rng.integers(0, 40)))
    N = int(p["cand_offsets"][-1])
    nsig = int(rng.integers(0, 5))
    sig = rng.integers(1, 6, nsig).tolist()  # repeats allowed: both thresholds must pass
    lt = rng.choice([-0.25, -0.5, -1.0, -1.5, -2.0, 0.0, -np.inf, np.inf], nsig).tolist()
    for budget in (0, 1, max(1, N // 3), N + 1):
        _log(f"[sparse] micro seed={seed} N={N} B={budget} sig={sig} lt={lt}")
        check(p["cand_offsets"], p["parent"], p["logq"], budget, sig, lt)


def test_many_small_and_empty_requests():
    """Blocks spanning more than 64 requests (score table overflow) and more than
    1024 requests with empty ones in between (truncation table overflow)."""
    rng = np.random.default_rng(4)
    R = 4000
    sizes = np.where(rng.random(R) < 0.6, 0, rng.integers(1, 5, R))
    offs = np.zeros(R + 1, np.int32)
    offs[1:] = np.cumsum(sizes)
    N = int(offs[-1])
    parent = np.empty(N, np.int32)
    for r in range(R):
        for n in range(int(sizes[r])):
            parent[offs[r] + n] = int(rng.integers(-1, n))
    logq = rng.choice(np.array([-0.25, -0.5, -1.0], np.float32), N)
    for budget in (100, 1500, N):
        _log(f"[sparse] many requests R={R} N={N} B={budget}")
        check(offs, parent, logq, budget, [1, 2], [-0.4, -0.9])


def test_no_checkpoints_reports_no_truncation():
    b = synth.make_batch("tiny", 3, attention=False)
    ref = check(b["cand_offsets"], b["parent"], b["logq"], b["cfg"].budget, [], [])
    assert np.all(ref["trunc_depth"] == st.MAX_DEPTH + 1)
    plain = oracle.gate(b["cand_offsets"], b["parent"], b["logq"], b["cfg"].budget)
    assert np.array_equal(ref["selected"], plain["selected"])


def test_full_step_with_sparse_gate():
    """The whole step (gate_sparse -> mask -> attention -> accept) on the tiny preset."""
    from paper_2604_09603_amd.step import VerifyStep
    b = synth.make_batch("tiny", 1)
    cfg = b["cfg"]
    sig, lt = [2, 3], _median_table(b, [2, 3])
    g = oracle.gate_sparse(b["cand_offsets"], b["parent"], b["logq"], cfg.budget, sig,
                           np.asarray(lt, np.float32))
    m = oracle.build_tree_mask(b["cand_offsets"], b["parent"], b["token"], g["selected"],
                               b["root_token"], b["prefix_len"], cfg.budget, cfg.mask_words)
    tgt = synth.target_for_slots(b, m["q_offsets"], m["slot_cand"])
    a = oracle.accept(m["q_offsets"], m["slot_parent"], m["slot_token"], tgt, 16)
    ro, rl, _ = oracle.tree_verify_attn(b["q"], b["k_new"], b["v_new"], b["k_cache"],
                                        b["v_cache"], b["kv_offsets"], m["q_offsets"],
                                        m["tree_mask"], cfg.hq, cfg.hkv, b["sm_scale"])
    stp = VerifyStep(b, checkpoints=list(zip(sig, lt)))
    stp.set_target(tgt)
    stp.run()
    res = stp.fetch()
    gc.compare_front(res, dict(gate=g, mask=m, accept=a), int(b["cand_offsets"][-1]))
    assert np.array_equal(res["trunc_depth"], g["trunc_depth"])
    gc.compare_attn(res["out"], res["lse"], ro, rl, range(m["num_slots"]))


@pytest.mark.parametrize("name", ["l8b", "q235b", "long"])
def test_ablation_dense_and_fixed_threshold(name):
    """The paper's ablation policies as checkpoint tables: dense gating (a
    checkpoint at every depth, thresholds at the median layer maximum) and a
    single fixed threshold at every depth."""
    b = synth.make_batch(name, 1, attention=False)
    depths = list(range(1, b["cfg"].depth + 1))
    dense = _median_table(b, depths)
    _log(f"[sparse] {name} dense gating {dense}")
    check(b["cand_offsets"], b["parent"], b["logq"], b["cfg"].budget, depths, dense)
    fixed = [dense[len(dense) // 2]] * len(depths)
    _log(f"[sparse] {name} fixed threshold {fixed[0]}")
    check(b["cand_offsets"], b["parent"], b["logq"], b["cfg"].budget, depths, fixed)
