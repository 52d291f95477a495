"""echo_verify_step (the four stages in one call, with the gate's last phase, the
mask and the attention plan in one launch) against the four separate calls on
the same inputs: every output bit for bit, status included, on the presets, the
narrow-head shapes and the adversarial micro batches; and one preset against the
oracle directly."""
import sys

import numpy as np
import pytest

import oracle
import synth
from tests import gpu_common as gc
from tests.test_gpu_edges import _front_ref, make_micro_batch

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _need_gpu():
    gc.require_gpu()


def _log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _run(batch, target, fused, repeat=1):
    import torch
    from paper_2604_09603_amd.step import VerifyStep
    st = VerifyStep(batch)
    st.out.fill_(float("nan"))
    st.lse.fill_(float("nan"))
    st.set_target(target)
    for _ in range(repeat):
        if fused:
            st.run_fused()
        else:
            st.run()
    res = st.fetch()
    torch.cuda.synchronize()
    return res


def _bits(x):
    a = np.ascontiguousarray(x)
    if a.dtype == np.float32:
        return a.view(np.uint32)
    return a


def _same(a, b):
    assert a.keys() == b.keys()
    for k in a:
        if isinstance(a[k], np.ndarray):
            assert a[k].shape == b[k].shape, k
            assert np.array_equal(_bits(a[k]), _bits(b[k])), f"{k} differs"
        else:
            assert a[k] == b[k], (k, a[k], b[k])


def _compare(batch, repeat=1):
    target = synth.target_for_slots(batch, *_slots(batch))
    sep = _run(batch, target, fused=False)
    fus = _run(batch, target, fused=True, repeat=repeat)
    _same(sep, fus)
    return fus


def _slots(batch):
    ref = _front_ref(batch)
    m = ref["mask"]
    return m["q_offsets"], m["slot_cand"]


@pytest.mark.parametrize("name,seed", [("tiny", s) for s in range(3)] +
                         [(n, 0) for n in ["l8b", "l70b", "q235b", "long", "q235b_tp4",
                                           "g1_decode", "g2_tree"]] +
                         [("q235b", 1), ("l70b", 2)])
def test_fused_step_equals_separate_calls(name, seed):
    _log(f"[fused] {name} seed={seed}")
    b = synth.make_batch(name, seed)
    res = _compare(b)
    assert res["status"] == 0


def test_fused_step_against_oracle():
    b = synth.make_batch("tiny", 7)
    ref = gc.oracle_front(b)
    res = _run(b, ref["target"], fused=True)
    gc.compare_front(res, ref, int(b["cand_offsets"][-1]))
    m = ref["mask"]
    cfg = b["cfg"]
    rows = list(range(m["num_slots"]))
    ro, rl, _ = oracle.tree_verify_attn(b["q"], b["k_new"], b["v_new"], b["k_cache"],
                                        b["v_cache"], b["kv_offsets"], m["q_offsets"],
                                        m["tree_mask"], cfg.hq, cfg.hkv, b["sm_scale"])
    gc.compare_attn(res["out"], res["lse"], ro, rl, rows)


def test_fused_step_repeated_calls():
    """The workspaces keep the previous call's contents: three calls in a row give
    the separate calls' outputs."""
    b = synth.make_batch("l8b", 4)
    _compare(b, repeat=3)


@pytest.mark.parametrize("budget", [0, 7, 500])
def test_fused_step_micro_pools(budget):
    rng = np.random.default_rng(40 + budget)
    pool = synth.micro_pool(rng, 300, 9, p_neg_inf=0.05)
    _log(f"[fused] micro B={budget}")
    _compare(make_micro_batch(pool, budget, hq=8, hkv=2, p_range=(0, 70), seed=budget))


def test_fused_step_maximum_sizes():
    """R = 4095 and B = 16384: the front kernel's LDS is at its largest (the mask's
    tables above the gate's candidate arrays)."""
    rng = np.random.default_rng(17)
    pool = synth.micro_pool(rng, 4095, 9, p_neg_inf=0.05)
    _log("[fused] max sizes")
    _compare(make_micro_batch(pool, 16384, hq=8, hkv=2, p_range=(0, 40), seed=5))


def test_fused_step_invalid_data_and_empty_requests():
    offs = np.array([0, 5, 9], np.int32)
    parent = np.array([-1, 0, 7, 1, 2, -1, -5, 0, 2], np.int32)
    logq = np.array([-0.5, np.nan, 0.25, -1.0, -0.5, -0.25, -0.5, -1.0, -2.0], np.float32)
    pool = dict(cand_offsets=offs, parent=parent, token=np.arange(9, dtype=np.int32) % 4,
                logq=logq, root_token=np.array([1, 2], np.int32))
    res = _compare(make_micro_batch(pool, 6, p_range=(3, 9)))
    assert (res["status"] & 7) == 7
    empty = dict(cand_offsets=np.zeros(4, np.int32), parent=np.zeros(0, np.int32),
                 token=np.zeros(0, np.int32), logq=np.zeros(0, np.float32),
                 root_token=np.array([1, 2, 3], np.int32))
    res = _compare(make_micro_batch(empty, 4, hq=8, hkv=4, p_range=(0, 50)))
    assert res["num_slots"] == 3
    offs = np.array([0, 0, 4, 4, 7], np.int32)
    parent = np.array([-1, 0, 0, 1, -1, -1, 1], np.int32)
    pool = dict(cand_offsets=offs, parent=parent, token=np.arange(7, dtype=np.int32) % 3,
                logq=np.array([-0.1, -0.2, -0.3, -0.4, -0.1, -0.5, -0.2], np.float32),
                root_token=np.array([0, 1, 2, 0], np.int32))
    _compare(make_micro_batch(pool, 5, hq=8, hkv=4, p_range=(0, 0)))


def test_fused_step_long_requests():
    """Requests with more verify slots than the tail kernel stages in LDS (256):
    its acceptance reads them from memory, the acceptance launch from LDS."""
    rng = np.random.default_rng(23)
    pool = synth.micro_pool(rng, 3, 700, p_neg_inf=0.0)
    _log("[fused] long requests")
    res = _compare(make_micro_batch(pool, 1200, hq=8, hkv=2, p_range=(0, 40), seed=9))
    assert int(np.diff(res["q_offsets"]).max()) > 256
