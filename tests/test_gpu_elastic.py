"""GPU parity of the elastic budget scheduler (Alg. 1): echo_gate_elastic
against oracle.elastic_schedule, bit for bit (path scores, selection, count,
truncation depths, status)."""
import sys

import numpy as np
import pytest

import oracle
import synth
from tests import gpu_common as gc

pytestmark = pytest.mark.gpu

PAPER_TAU = {"l8b": {1: 0.2, 5: 0.35, 8: 0.5}, "q235b": {1: 0.15, 3: 0.3, 5: 0.5}}


@pytest.fixture(autouse=True)
def _need_gpu():
    gc.require_gpu()


def _log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def run_elastic(offs, parent, logq, budget, sig, log_tau, w_topk, w_max):
    import torch
    import paper_2604_09603_amd as pkg
    from paper_2604_09603_amd.step import _aligned_workspace
    d = "cuda:0"
    R, N = len(offs) - 1, int(offs[-1])
    t = lambda a, dt: torch.from_numpy(np.ascontiguousarray(a).astype(dt)).to(d)
    path = torch.full((max(N, 1),), float("nan"), dtype=torch.float32, device=d)
    sel = torch.full((max(N, 1),), 7, dtype=torch.uint8, device=d)
    nsel = torch.full((1,), -1, dtype=torch.int32, device=d)
    trunc = torch.full((R,), -5, dtype=torch.int32, device=d)
    status = torch.zeros(1, dtype=torch.int32, device=d)
    ws = _aligned_workspace(pkg.gate_elastic_workspace_size(R, N, budget), d)
    ws.fill_(0xCD)  # the workspace's contents on entry must not matter
    pkg.echo_gate_elastic(t(offs, np.int32), t(parent, np.int32), t(logq, np.float32), R, N,
                          budget, sig, log_tau, w_topk, w_max, path, sel, nsel, ws,
                          trunc_depth=trunc, status=status)
    torch.cuda.synchronize()
    return dict(path_score=path.cpu().numpy()[:N], selected=sel.cpu().numpy()[:N],
                num_selected=int(nsel.item()), status=int(status.item()),
                trunc_depth=trunc.cpu().numpy())


def check(offs, parent, logq, budget, sig, log_tau, w_topk, w_max):
    lt = np.asarray(log_tau, np.float32)
    ref = oracle.elastic_schedule(offs, parent, logq, budget, list(sig), lt, w_topk, w_max)
    got = run_elastic(offs, parent, logq, budget, list(sig), lt.tolist(), w_topk, w_max)
    assert np.array_equal(got["path_score"].view(np.uint32), ref["path_score"].view(np.uint32))
    assert np.array_equal(got["selected"], ref["selected"]), "selection differs"
    assert got["num_selected"] == ref["num_selected"]
    assert np.array_equal(got["trunc_depth"], ref["trunc_depth"]), "truncation depths differ"
    assert got["status"] == ref["status"]
    return ref


def _median_table(b, depths):
    from oracle.gate import layer_max_scores
    S, depth, _ = oracle.path_scores(b["cand_offsets"], b["parent"], b["logq"])
    lm = layer_max_scores(b["cand_offsets"], S, depth)
    return [float(np.float32(np.median(lm[:, d]))) for d in depths]


@pytest.mark.parametrize("name,seed", [(n, s) for n in ["tiny", "l8b", "l70b", "q235b", "long"]
                                       for s in (0, 1)])
def test_presets(name, seed):
    """Checkpoints at depths 1, 3, 5 at the median layer maximum, three widths."""
    b = synth.make_batch(name, seed, attention=False)
    sig = [1, 3, 5]
    lt = _median_table(b, sig)
    k = b["cfg"].branch
    for wt, wm in [(1, 3), (2, k), (k, 2 * k)]:
        _log(f"[elastic] {name} seed={seed} w_topk={wt} w_max={wm}")
        check(b["cand_offsets"], b["parent"], b["logq"], b["cfg"].budget, sig, lt, wt, wm)


@pytest.mark.parametrize("name", sorted(PAPER_TAU))
def test_paper_thresholds_and_large_budgets(name):
    b = synth.make_batch(name, 2, attention=False)
    tab = PAPER_TAU[name]
    sig = sorted(tab)
    lt = [float(np.log(np.float32(tab[d]))) for d in sig]
    N = int(b["cand_offsets"][-1])
    for budget in (b["cfg"].budget, 4 * b["cfg"].budget, min(N, 16384)):  # 16384: budget limit
        _log(f"[elastic] {name} paper table B={budget}")
        check(b["cand_offsets"], b["parent"], b["logq"], budget, sig, lt, 2, 6)


@pytest.mark.parametrize("seed", range(16))
def test_micro_pools_with_ties(seed):
    rng = np.random.default_rng(1300 + seed)
    p = synth.micro_pool(rng, int(rng.integers(1, 7)), int(rng.integers(0, 40)))
    N = int(p["cand_offsets"][-1])
    nsig = int(rng.integers(0, 4))
    sig = rng.integers(1, 6, nsig).tolist()
    lt = rng.choice([-0.25, -0.5, -1.0, -1.5, 0.0, -np.inf], nsig).tolist()
    wt, wm = int(rng.integers(1, 4)), int(rng.integers(0, 7))
    for budget in (0, 1, max(1, N // 3), N + 1):
        _log(f"[elastic] micro seed={seed} N={N} B={budget} sig={sig} lt={lt} w={wt},{wm}")
        check(p["cand_offsets"], p["parent"], p["logq"], budget, sig, lt, wt, wm)


def test_requests_larger_than_lds():
    """Requests of 5000 and 9000 candidates: their trajectories run from the
    workspace instead of LDS."""
    rng = np.random.default_rng(8)
    sizes = [5000, 30, 9000]
    offs = np.zeros(len(sizes) + 1, np.int32)
    offs[1:] = np.cumsum(sizes)
    parent = np.concatenate([np.array([-1] + [int(rng.integers(-1, n)) for n in range(1, s)],
                                      np.int32) for s in sizes])
    logq = rng.choice(np.array([-0.25, -0.5, -1.0, -2.0], np.float32), int(offs[-1]))
    for budget, wt, wm in [(40, 3, 9), (700, 50, 120), (16000, 4000, 8000)]:
        _log(f"[elastic] large requests B={budget} w={wt},{wm}")
        check(offs, parent, logq, budget, [2, 4], [-1.0, -2.6], wt, wm)


def test_many_small_requests():
    rng = np.random.default_rng(9)
    R = 3000
    sizes = np.where(rng.random(R) < 0.3, 0, rng.integers(1, 6, R))
    offs = np.zeros(R + 1, np.int32)
    offs[1:] = np.cumsum(sizes)
    N = int(offs[-1])
    parent = np.empty(N, np.int32)
    for r in range(R):
        for n in range(int(sizes[r])):
            parent[offs[r] + n] = int(rng.integers(-1, n))
    logq = rng.choice(np.array([-0.25, -0.5, -1.0], np.float32), N)
    for budget in (1000, 2500, N):
        _log(f"[elastic] many requests R={R} N={N} B={budget}")
        check(offs, parent, logq, budget, [2], [-0.9], 2, 3)


def test_full_step_with_elastic_gate():
    from paper_2604_09603_amd.step import VerifyStep
    b = synth.make_batch("tiny", 2)
    cfg = b["cfg"]
    sig, lt = [2, 3], _median_table(b, [2, 3])
    g = oracle.elastic_schedule(b["cand_offsets"], b["parent"], b["logq"], cfg.budget, sig,
                                np.asarray(lt, np.float32), 2, 4)
    m = oracle.build_tree_mask(b["cand_offsets"], b["parent"], b["token"], g["selected"],
                               b["root_token"], b["prefix_len"], cfg.budget, cfg.mask_words)
    tgt = synth.target_for_slots(b, m["q_offsets"], m["slot_cand"])
    a = oracle.accept(m["q_offsets"], m["slot_parent"], m["slot_token"], tgt, 16)
    ro, rl, _ = oracle.tree_verify_attn(b["q"], b["k_new"], b["v_new"], b["k_cache"],
                                        b["v_cache"], b["kv_offsets"], m["q_offsets"],
                                        m["tree_mask"], cfg.hq, cfg.hkv, b["sm_scale"])
    stp = VerifyStep(b, checkpoints=list(zip(sig, lt)), elastic=(2, 4))
    stp.set_target(tgt)
    stp.run()
    res = stp.fetch()
    gc.compare_front(res, dict(gate=g, mask=m, accept=a), int(b["cand_offsets"][-1]))
    assert np.array_equal(res["trunc_depth"], g["trunc_depth"])
    gc.compare_attn(res["out"], res["lse"], ro, rl, range(m["num_slots"]))
