"""Shared pieces of the GPU parity tests: run the library and the oracle on one batch."""
import functools
import math

import numpy as np
import pytest

import oracle
import synth

ATOL = 1e-2       # max-abs error of attention outputs
RTOL_ROW = 1e-2   # per-(slot, head) normwise relative error
LSE_ATOL = 1e-3


def gpu_available():
    try:
        import torch
        return torch.cuda.is_available()
    except Exception:
        return False


def require_gpu():
    if not gpu_available():
        pytest.skip("no GPU")


def oracle_front(batch):
    """Oracle gate + mask + accept (all integer/fp32-exact stages) on a batch."""
    cfg = batch["cfg"]
    g = oracle.gate(batch["cand_offsets"], batch["parent"], batch["logq"], cfg.budget)
    m = oracle.build_tree_mask(batch["cand_offsets"], batch["parent"], batch["token"],
                               g["selected"], batch["root_token"], batch["prefix_len"],
                               cfg.budget, cfg.mask_words)
    tgt = synth.target_for_slots(batch, m["q_offsets"], m["slot_cand"])
    a = oracle.accept(m["q_offsets"], m["slot_parent"], m["slot_token"], tgt, 16)
    return dict(gate=g, mask=m, target=tgt, accept=a)


def run_gpu(batch, target, repeat=1):
    import torch
    from paper_2604_09603_amd.step import VerifyStep
    st = VerifyStep(batch)
    st.out.fill_(float("nan"))
    st.lse.fill_(float("nan"))
    st.set_target(target)
    res = None
    for _ in range(repeat):
        st.run()
        res = st.fetch()
    torch.cuda.synchronize()
    return st, res


def compare_front(res, ref, N):
    g, m, a = ref["gate"], ref["mask"], ref["accept"]
    assert np.array_equal(res["path_score"].view(np.uint32), g["path_score"].view(np.uint32)), \
        "path scores differ"
    assert np.array_equal(res["selected"], g["selected"]), "selection differs"
    assert res["num_selected"] == g["num_selected"]
    nq = m["num_slots"]
    assert res["num_slots"] == nq
    assert np.array_equal(res["q_offsets"], m["q_offsets"])
    for k in ["slot_cand", "slot_parent", "slot_token", "position_ids"]:
        assert np.array_equal(res[k][:nq], m[k][:nq]), k
    assert np.array_equal(res["tree_mask"][:nq], m["tree_mask"][:nq]), "tree mask differs"
    assert np.array_equal(res["accept_len"], a["accept_len"])
    assert np.array_equal(res["accept_slots"], a["accept_slots"])
    assert np.array_equal(res["bonus_token"], a["bonus_token"])


def compare_attn(out, lse, ref_out, ref_lse, rows):
    rows = list(rows)
    o, r = out[rows].astype(np.float64), ref_out[rows]
    l, rl = lse[rows].astype(np.float64), ref_lse[rows]
    empty = np.isneginf(rl)
    assert np.array_equal(np.isneginf(l), empty), "rows without keys differ"
    assert np.all(o[empty] == 0.0)
    diff = np.abs(o - r)
    assert diff.max() <= ATOL, f"max abs error {diff.max():.3e}"
    scale = np.maximum(np.abs(r).max(axis=-1), 1e-6)
    rel = diff.max(axis=-1) / scale
    assert rel.max() <= RTOL_ROW, f"row-relative error {rel.max():.3e}"
    fin = ~empty
    if fin.any():
        assert np.abs(l[fin] - rl[fin]).max() <= LSE_ATOL
    return float(diff.max()), float(rel.max())


def sample_rows(q_offsets, rng, n_requests=4, n_extra=48):
    """All slots of a few requests plus a few random slots."""
    R = len(q_offsets) - 1
    nq = int(q_offsets[-1])
    reqs = rng.choice(R, size=min(n_requests, R), replace=False)
    rows = set()
    for r in reqs:
        rows.update(range(int(q_offsets[r]), int(q_offsets[r + 1])))
    rows.update(rng.choice(nq, size=min(n_extra, nq), replace=False).tolist())
    return sorted(rows)
