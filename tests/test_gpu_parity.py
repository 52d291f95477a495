"""GPU parity: libecho (HIP, gfx950) against the CPU oracle on the same seeded inputs.

Gate, mask and accept outputs must match bit for bit; attention must satisfy
max-abs <= 1e-2, per-row normwise relative <= 1e-2 and LSE within 1e-3 of
the float64 oracle.
"""
import sys

import numpy as np
import pytest

import oracle
import synth
from tests import gpu_common as gc

pytestmark = pytest.mark.gpu


def _log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(autouse=True)
def _need_gpu():
    gc.require_gpu()


def _attn_ref(batch, m, rows):
    cfg = batch["cfg"]
    out, lse, st = oracle.tree_verify_attn(batch["q"], batch["k_new"], batch["v_new"],
                                           batch["k_cache"], batch["v_cache"], batch["kv_offsets"],
                                           m["q_offsets"], m["tree_mask"], cfg.hq, cfg.hkv,
                                           batch["sm_scale"], rows=rows)
    return out, lse


@pytest.mark.parametrize("name,seed", [("tiny", s) for s in range(5)] +
                         [(n, s) for n in ["l8b", "l70b", "q235b", "long"] for s in range(5)])
def test_presets_match_oracle(name, seed):
    _log(f"[parity] {name} seed={seed}: generating")
    b = synth.make_batch(name, seed)
    ref = gc.oracle_front(b)
    _log(f"[parity] {name} seed={seed}: gpu run")
    st, res = gc.run_gpu(b, ref["target"])
    gc.compare_front(res, ref, int(b["cand_offsets"][-1]))
    assert res["status"] == 0
    m = ref["mask"]
    rng = np.random.default_rng(seed)
    rows = list(range(m["num_slots"])) if name == "tiny" else gc.sample_rows(m["q_offsets"], rng)
    _log(f"[parity] {name} seed={seed}: oracle attention on {len(rows)} slots")
    ro, rl = _attn_ref(b, m, rows)
    err = gc.compare_attn(res["out"], res["lse"], ro, rl, rows)
    # rows beyond the verified slots are never written
    nq = m["num_slots"]
    assert np.all(np.isnan(res["out"][nq:])) and np.all(np.isnan(res["lse"][nq:]))
    _log(f"[parity] {name} seed={seed}: ok, attention max abs {err[0]:.2e}, row rel {err[1]:.2e}")


@pytest.mark.parametrize("name", ["g1_decode", "g1_tree", "g2_tree", "q235b_tp4"])
def test_narrow_groups_match_oracle(name):
    """GQA groups of one and two query heads (one row per stream in decode):
    streams with fewer rows than one matrix tile; and one KV head with a group of
    16 (a TP-4 share of the Qwen3-235B-shaped batch): fewer streams per request than
    a unit has waves.  Sampled rows against the oracle."""
    _log(f"[parity] {name}: generating")
    b = synth.make_batch(name, 2)
    ref = gc.oracle_front(b)
    st, res = gc.run_gpu(b, ref["target"])
    gc.compare_front(res, ref, int(b["cand_offsets"][-1]))
    m = ref["mask"]
    rows = gc.sample_rows(m["q_offsets"], np.random.default_rng(2), n_requests=6, n_extra=64)
    ro, rl = _attn_ref(b, m, rows)
    err = gc.compare_attn(res["out"], res["lse"], ro, rl, rows)
    _log(f"[parity] {name}: ok, attention max abs {err[0]:.2e}, row rel {err[1]:.2e}")


@pytest.mark.parametrize("name", ["tiny", "l8b", "l70b", "q235b", "long"])
def test_peaked_queries(name):
    """Queries scaled x4: sharper softmax, outputs of order one."""
    b = synth.make_batch(name, 7, q_scale=4.0)
    ref = gc.oracle_front(b)
    st, res = gc.run_gpu(b, ref["target"])
    gc.compare_front(res, ref, int(b["cand_offsets"][-1]))
    m = ref["mask"]
    rows = gc.sample_rows(m["q_offsets"], np.random.default_rng(3))
    ro, rl = _attn_ref(b, m, rows)
    gc.compare_attn(res["out"], res["lse"], ro, rl, rows)


@pytest.mark.parametrize("name", ["tiny", "l8b", "l70b", "q235b", "long"])
def test_scaled_values(name):
    """Values (new and cached) scaled x4, plain and with queries also scaled x4
    (outputs of order four, weight on fewer keys): sampled rows of every preset,
    every row of tiny and of l8b (160 slots x 32 heads), at the same absolute
    bounds."""
    for q_scale in (1.0, 4.0):
        b = synth.make_batch(name, 11, q_scale=q_scale, v_scale=4.0)
        ref = gc.oracle_front(b)
        st, res = gc.run_gpu(b, ref["target"])
        gc.compare_front(res, ref, int(b["cand_offsets"][-1]))
        m = ref["mask"]
        rows = (list(range(m["num_slots"])) if name in ("tiny", "l8b") else
                gc.sample_rows(m["q_offsets"], np.random.default_rng(5)))
        ro, rl = _attn_ref(b, m, rows)
        err = gc.compare_attn(res["out"], res["lse"], ro, rl, rows)
        _log(f"[parity] {name} V x4, Q x{q_scale:g}: max abs {err[0]:.2e}, row rel {err[1]:.2e}")


def test_repeat_is_bit_identical():
    b = synth.make_batch("l8b", 3)
    ref = gc.oracle_front(b)
    st, first = gc.run_gpu(b, ref["target"])
    st.run()
    second = st.fetch()
    for k in ["out", "lse", "selected", "tree_mask", "accept_len", "path_score"]:
        assert np.array_equal(np.asarray(first[k]).view(np.uint8), np.asarray(second[k]).view(np.uint8)), k


@pytest.mark.parametrize("name", ["l8b", "q235b"])
def test_large_values_through_cut_units(name):
    """Values scaled by 2^14 (outputs of order 10^4, far past the fp16 range once
    summed over a workgroup's keys): the partials of units cut between
    workgroups are stored in fp16 with a power-of-two scale per row, so the
    merged rows stay finite and within the row-relative bound, like the rows
    written directly.  Every slot of 8 requests plus 256 random slots."""
    b = synth.make_batch(name, 13, v_scale=float(2 ** 14))
    ref = gc.oracle_front(b)
    st, res = gc.run_gpu(b, ref["target"])
    gc.compare_front(res, ref, int(b["cand_offsets"][-1]))
    m = ref["mask"]
    rows = gc.sample_rows(m["q_offsets"], np.random.default_rng(6), n_requests=8, n_extra=256)
    ro, rl = _attn_ref(b, m, rows)
    ro, rl = ro[rows], rl[rows]
    o = res["out"][rows].astype(np.float64)
    assert np.isfinite(o).all(), "non-finite output rows"
    scale = np.maximum(np.abs(ro).max(axis=-1), 1e-6)
    rel = (np.abs(o - ro).max(axis=-1) / scale).max()
    _log(f"[parity] {name} V x2^14: row rel {rel:.2e}, largest output {np.abs(ro).max():.3e}")
    assert rel <= gc.RTOL_ROW, f"row-relative error {rel:.3e}"
    assert np.abs(res["lse"][rows] - rl).max() <= gc.LSE_ATOL
