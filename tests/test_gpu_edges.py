"""GPU parity on small adversarial inputs: score ties, degenerate budgets, empty
requests, empty prefixes, invalid data (status bits), deep chains, wide masks."""
import math
import sys

import numpy as np
import pytest

import oracle
import synth
from tests import gpu_common as gc

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _need_gpu():
    gc.require_gpu()


def _bf16(rng, *shape, scale=1.0):
    return synth.f32_to_bf16_bits(rng.standard_normal(shape).astype(np.float32) * np.float32(scale))


def make_micro_batch(pool, budget, hq=8, hkv=2, p_range=(0, 70), seed=0, v_scale=1.0):
    """Wrap a candidate pool into a full batch with random attention tensors
    (values multiplied by v_scale and rounded back to bf16)."""
    rng = np.random.default_rng(seed)
    R = len(pool["cand_offsets"]) - 1
    cfg = synth.Config("micro", R, 1, 1, 1.0, 8, budget, hq, hkv, 128, p_range[0], p_range[1],
                       ("const", 1.0))
    P = rng.integers(p_range[0], p_range[1] + 1, size=R).astype(np.int32)
    kvo = np.zeros(R + 1, np.int64)
    kvo[1:] = np.cumsum(P)
    T = int(kvo[-1])
    cap = R + budget
    N = int(pool["cand_offsets"][-1])
    b = dict(cfg=cfg, seed=seed, cand_offsets=pool["cand_offsets"].astype(np.int32),
             parent=pool["parent"].astype(np.int32), token=pool["token"].astype(np.int32),
             logq=pool["logq"].astype(np.float32), root_token=pool["root_token"].astype(np.int32),
             target=rng.integers(0, 4, size=N).astype(np.int32),
             root_target=rng.integers(0, 4, size=R).astype(np.int32),
             prefix_len=P, kv_offsets=kvo, q=_bf16(rng, cap, hq, 128),
             k_new=_bf16(rng, cap, hkv, 128), v_new=_bf16(rng, cap, hkv, 128, scale=v_scale),
             k_cache=_bf16(rng, T, hkv, 128), v_cache=_bf16(rng, T, hkv, 128, scale=v_scale),
             sm_scale=np.float32(1 / math.sqrt(128)))
    return b


def _front_ref(b, max_depth=16):
    cfg = b["cfg"]
    g = oracle.gate(b["cand_offsets"], b["parent"], b["logq"], cfg.budget)
    m = oracle.build_tree_mask(b["cand_offsets"], b["parent"], b["token"], g["selected"],
                               b["root_token"], b["prefix_len"], cfg.budget, cfg.mask_words)
    tgt = synth.target_for_slots(b, m["q_offsets"], m["slot_cand"])
    a = oracle.accept(m["q_offsets"], m["slot_parent"], m["slot_token"], tgt, max_depth)
    return dict(gate=g, mask=m, target=tgt, accept=a,
                status=g["status"] | m["status"] | a["status"])


def _check_all(b, attention=True):
    ref = _front_ref(b)
    st, res = gc.run_gpu(b, ref["target"])
    gc.compare_front(res, ref, int(b["cand_offsets"][-1]))
    assert res["status"] == ref["status"], (res["status"], ref["status"])
    if attention:
        cfg = b["cfg"]
        m = ref["mask"]
        rows = list(range(m["num_slots"]))
        ro, rl, _ = oracle.tree_verify_attn(b["q"], b["k_new"], b["v_new"], b["k_cache"],
                                            b["v_cache"], b["kv_offsets"], m["q_offsets"],
                                            m["tree_mask"], cfg.hq, cfg.hkv, b["sm_scale"])
        gc.compare_attn(res["out"], res["lse"], ro, rl, rows)
    return res, ref


@pytest.mark.parametrize("seed", range(24))
def test_micro_pools_with_ties(seed):
    rng = np.random.default_rng(1000 + seed)
    pool = synth.micro_pool(rng, int(rng.integers(1, 7)), int(rng.integers(0, 40)), vocab=4)
    N = int(pool["cand_offsets"][-1])
    budget = int(rng.choice([0, 1, 3, max(1, N // 3), N, N + 5]))
    hq, hkv = [(8, 2), (4, 4), (16, 1), (6, 3)][seed % 4]
    b = make_micro_batch(pool, budget, hq, hkv, p_range=(0, 150), seed=seed)
    print(f"[edges] micro seed={seed} R={len(pool['cand_offsets']) - 1} N={N} B={budget}", flush=True)
    _check_all(b)


def test_invalid_data_sets_status_bits():
    offs = np.array([0, 5, 9], np.int32)
    parent = np.array([-1, 0, 7, 1, 2, -1, -5, 0, 2], np.int32)      # 7 and -5 are bad
    logq = np.array([-0.5, np.nan, 0.25, -1.0, -0.5, -0.25, -0.5, -1.0, -2.0], np.float32)
    pool = dict(cand_offsets=offs, parent=parent, token=np.arange(9, dtype=np.int32) % 4,
                logq=logq, root_token=np.array([1, 2], np.int32))
    b = make_micro_batch(pool, 6, p_range=(3, 9))
    res, ref = _check_all(b)
    assert (res["status"] & 7) == 7


@pytest.mark.parametrize("offs", [[2, 5, 9], [0, 6, 4, 9]])
def test_malformed_candidate_csr(offs):
    """A candidate CSR that does not start at 0 or decreases: nothing is scored or
    packed, every request keeps its root slot, and BAD_OFFSETS is raised."""
    offs = np.array(offs, np.int32)
    R = len(offs) - 1
    parent = np.array([-1, 0, 1, -1, 3, -1, 5, 6, -1], np.int32)
    pool = dict(cand_offsets=offs, parent=parent, token=np.arange(9, dtype=np.int32) % 4,
                logq=np.full(9, -0.5, np.float32), root_token=np.arange(R, dtype=np.int32))
    print(f"[edges] malformed csr {offs.tolist()}", flush=True)
    b = make_micro_batch(pool, 4, p_range=(3, 40))
    res, ref = _check_all(b)
    assert res["status"] & oracle.status.BAD_OFFSETS
    assert res["num_slots"] == R


def test_deep_chain_and_wide_mask():
    """A 20-deep chain (depth cap) plus 70 root children in another request (3 mask words)."""
    p1 = np.array([-1] + list(range(19)), np.int32)
    p2 = np.full(70, -1, np.int32)
    pool = dict(cand_offsets=np.array([0, 20, 90], np.int32), parent=np.concatenate([p1, p2]),
                token=np.zeros(90, np.int32), logq=np.full(90, -0.001, np.float32),
                root_token=np.array([0, 0], np.int32))
    b = make_micro_batch(pool, 80, hq=4, hkv=4, p_range=(0, 40))
    res, ref = _check_all(b)
    assert res["status"] & 8


def test_all_equal_scores_large_tie_class():
    """Thousands of candidates with identical path scores: ties resolved by index."""
    rng = np.random.default_rng(5)
    R, n = 6, 1500
    offs = np.arange(R + 1, dtype=np.int32) * n
    parent = np.concatenate([np.array([-1] * 40 + [int(rng.integers(0, 40)) for _ in range(n - 40)],
                                      np.int32) for _ in range(R)])
    pool = dict(cand_offsets=offs, parent=parent, token=np.zeros(R * n, np.int32),
                logq=np.full(R * n, -0.5, np.float32), root_token=np.zeros(R, np.int32))
    for budget in (100, 239, 240, 241, 5000):
        b = make_micro_batch(pool, budget, hq=4, hkv=2, p_range=(10, 20))
        _check_all(b, attention=(budget == 241))


def test_crowded_threshold_bin():
    """20k distinct path scores inside one 11-bit key bin: the threshold is found
    over more keys than the finish kernel gathers into LDS, and at budgets whose
    boundary falls inside the bin."""
    rng = np.random.default_rng(11)
    R, n = 4, 5000
    offs = np.arange(R + 1, dtype=np.int32) * n
    parent = np.full(R * n, -1, np.int32)
    logq = rng.uniform(-0.99, -0.88, R * n).astype(np.float32)
    pool = dict(cand_offsets=offs, parent=parent, token=np.zeros(R * n, np.int32),
                logq=logq, root_token=np.zeros(R, np.int32))
    for budget in (1, 700, 4097, 12345):
        print(f"[edges] crowded bin B={budget}", flush=True)
        b = make_micro_batch(pool, budget, hq=4, hkv=2, p_range=(10, 20))
        _check_all(b, attention=False)


@pytest.mark.parametrize("budget", [5000, 16384])
def test_maximum_batch_and_budget(budget):
    """R = 4095 requests (the limit; the attention plan takes its multi-pass
    path beyond 256) with up to 9 candidates each, budgets up to 16384 (the
    limit: 513 mask words per slot)."""
    rng = np.random.default_rng(17)
    pool = synth.micro_pool(rng, 4095, 9, p_neg_inf=0.05)
    N = int(pool["cand_offsets"][-1])
    print(f"[edges] max sizes R=4095 N={N} B={budget}", flush=True)
    b = make_micro_batch(pool, budget, hq=8, hkv=2, p_range=(0, 40), seed=5)
    ref = _front_ref(b)
    st, res = gc.run_gpu(b, ref["target"])
    gc.compare_front(res, ref, N)
    assert res["status"] == ref["status"]
    cfg = b["cfg"]
    m = ref["mask"]
    # every row: with prefixes of at most 40 keys many rows put their weight on
    # a few keys, where the rounding of the probabilities to bf16 shows most
    ro, rl, _ = oracle.tree_verify_attn(b["q"], b["k_new"], b["v_new"], b["k_cache"],
                                        b["v_cache"], b["kv_offsets"], m["q_offsets"],
                                        m["tree_mask"], cfg.hq, cfg.hkv, b["sm_scale"])
    err = gc.compare_attn(res["out"], res["lse"], ro, rl, range(m["num_slots"]))
    print(f"[edges] max sizes B={budget}: max abs {err[0]:.2e}, row rel {err[1]:.2e}", flush=True)


@pytest.mark.parametrize("seed", range(4))
def test_few_key_rows_every_row(seed):
    """Rows over short prefixes (0-40 keys) and small trees, all of them
    checked: a row whose softmax weight sits on one or two keys is the worst
    case for the bf16 probabilities of the P V product."""
    rng = np.random.default_rng(300 + seed)
    pool = synth.micro_pool(rng, 1024, 9, p_neg_inf=0.05)
    b = make_micro_batch(pool, 2000, hq=8, hkv=2, p_range=(0, 40), seed=seed)
    ref = _front_ref(b)
    st, res = gc.run_gpu(b, ref["target"])
    gc.compare_front(res, ref, int(b["cand_offsets"][-1]))
    cfg = b["cfg"]
    m = ref["mask"]
    ro, rl, _ = oracle.tree_verify_attn(b["q"], b["k_new"], b["v_new"], b["k_cache"],
                                        b["v_cache"], b["kv_offsets"], m["q_offsets"],
                                        m["tree_mask"], cfg.hq, cfg.hkv, b["sm_scale"])
    err = gc.compare_attn(res["out"], res["lse"], ro, rl, range(m["num_slots"]))
    print(f"[edges] few keys, seed {seed}: max abs {err[0]:.2e}, row rel {err[1]:.2e}", flush=True)


@pytest.mark.parametrize("seed", range(2))
def test_few_key_rows_scaled_values_every_row(seed):
    """The few-key batches with every value multiplied by 4: the bf16 rounding of
    the probabilities moves the output by a fraction of the spread of the values
    that carry the weight, so this is where the absolute 1e-2 bound is tightest."""
    rng = np.random.default_rng(300 + seed)
    pool = synth.micro_pool(rng, 1024, 9, p_neg_inf=0.05)
    b = make_micro_batch(pool, 2000, hq=8, hkv=2, p_range=(0, 40), seed=seed, v_scale=4.0)
    ref = _front_ref(b)
    st, res = gc.run_gpu(b, ref["target"])
    cfg = b["cfg"]
    m = ref["mask"]
    ro, rl, _ = oracle.tree_verify_attn(b["q"], b["k_new"], b["v_new"], b["k_cache"],
                                        b["v_cache"], b["kv_offsets"], m["q_offsets"],
                                        m["tree_mask"], cfg.hq, cfg.hkv, b["sm_scale"])
    err = gc.compare_attn(res["out"], res["lse"], ro, rl, range(m["num_slots"]))
    print(f"[edges] few keys, V x4, seed {seed}: max abs {err[0]:.2e}, row rel {err[1]:.2e}",
          flush=True)


@pytest.mark.parametrize("seed", range(2))
def test_late_dominant_key_every_row(seed):
    """A key in the last two tiles of a long prefix carries about 40% of every
    row's weight, and a key in the first prefix tile, one unit of log2 below
    it, about 20% (each request's queries are one vector per KV head; both keys
    are that vector scaled to the wanted logit; the other keys and the tree's
    keys have logits of order 0.25).  The early key raises the softmax
    reference, so the late key's probability is 2^(1 + e), not a power of two,
    and its bf16 rounding moves the output by up to 2^-9 of the value spread
    (6e-3 to 9e-3 on these batches) unless the residual product runs (3e-4).
    Rows of units cut between workgroups are merged from partials stored in
    fp16, each row scaled by a power of two: their rounding is 2^-12 of the
    row's largest value, up to 2e-3 here (values of V times 4).  The kernel
    screens the residual test with a threshold taken at earlier tiles; the bound
    of 3e-3 on every row shows the late tile still got through."""
    rng = np.random.default_rng(500 + seed)
    R, hq, hkv = 8, 32, 2
    G = hq // hkv
    pool = synth.micro_pool(rng, R, 9, p_neg_inf=0.0)
    b = make_micro_batch(pool, 24, hq=hq, hkv=hkv, p_range=(1800, 2600), seed=seed,
                         v_scale=4.0)
    scale = float(b["sm_scale"])
    kf = synth.bf16_bits_to_f32(b["k_cache"]) * np.float32(0.25)
    kn = synth.bf16_bits_to_f32(b["k_new"]) * np.float32(0.25)
    q = synth.bf16_bits_to_f32(b["q"])
    P, kvo = b["prefix_len"], b["kv_offsets"]
    qo = _front_ref(b)["mask"]["q_offsets"]   # the slots do not depend on q or k
    for r in range(R):
        early = int(kvo[r]) + int(rng.integers(0, 32))
        late = int(kvo[r]) + int(P[r]) - 1 - int(rng.integers(0, 64))
        for h in range(hkv):
            q0 = synth.bf16_bits_to_f32(
                synth.f32_to_bf16_bits(rng.standard_normal(128).astype(np.float32)))
            q[qo[r]:qo[r + 1], h * G:(h + 1) * G, :] = q0
            unit = q0 / np.float32(float(q0 @ q0) * scale)   # logit 1 (natural units)
            logit = math.log(float(P[r]))
            kf[late, h, :] = unit * np.float32(logit)
            kf[early, h, :] = unit * np.float32(logit - math.log(2.0))
    b["q"] = synth.f32_to_bf16_bits(q)
    b["k_cache"] = synth.f32_to_bf16_bits(kf)
    b["k_new"] = synth.f32_to_bf16_bits(kn)
    ref = _front_ref(b)
    st, res = gc.run_gpu(b, ref["target"])
    gc.compare_front(res, ref, int(b["cand_offsets"][-1]))
    cfg = b["cfg"]
    m = ref["mask"]
    ro, rl, _ = oracle.tree_verify_attn(b["q"], b["k_new"], b["v_new"], b["k_cache"],
                                        b["v_cache"], b["kv_offsets"], m["q_offsets"],
                                        m["tree_mask"], cfg.hq, cfg.hkv, b["sm_scale"])
    nq = m["num_slots"]
    gc.compare_attn(res["out"], res["lse"], ro, rl, range(nq))
    err = np.abs(res["out"][:nq].astype(np.float64) - ro[:nq]).max()
    print(f"[edges] late dominant key, seed {seed}: max abs {err:.2e} over {nq * hq} rows",
          flush=True)
    assert err <= 3e-3, f"max abs error {err:.3e}: the late tile's residual product did not run"


def test_empty_requests_and_prefixes():
    offs = np.array([0, 0, 4, 4, 7], np.int32)            # requests 0 and 2 have no candidates
    parent = np.array([-1, 0, 0, 1, -1, -1, 1], np.int32)
    pool = dict(cand_offsets=offs, parent=parent, token=np.arange(7, dtype=np.int32) % 3,
                logq=np.array([-0.1, -0.2, -0.3, -0.4, -0.1, -0.5, -0.2], np.float32),
                root_token=np.array([0, 1, 2, 0], np.int32))
    b = make_micro_batch(pool, 5, hq=8, hkv=4, p_range=(0, 0))    # no KV prefix at all
    _check_all(b)
    b = make_micro_batch(pool, 0, hq=8, hkv=4, p_range=(0, 300))  # budget 0: decode only
    _check_all(b)
    # no candidates in the whole batch (N = 0): every request verifies its root only
    empty = dict(cand_offsets=np.zeros(4, np.int32), parent=np.zeros(0, np.int32),
                 token=np.zeros(0, np.int32), logq=np.zeros(0, np.float32),
                 root_token=np.array([1, 2, 3], np.int32))
    b = make_micro_batch(empty, 4, hq=8, hkv=4, p_range=(0, 50))
    res, _ = _check_all(b)
    assert res["num_slots"] == 3


# (Hq, Hkv): one KV head (every stream of a unit is a pass of the same head),
# a KV-head count that is not a power of two, and wide GQA groups, so that the
# 4-stream units of the attention plan straddle heads and passes in every way
HEAD_LAYOUTS = [(1, 1), (8, 1), (32, 1), (6, 3), (15, 5), (12, 6), (56, 7), (64, 2), (96, 3)]


@pytest.mark.parametrize("hq,hkv", HEAD_LAYOUTS)
def test_head_layouts_every_row(hq, hkv):
    """Random trees (up to 30 candidates per request, so up to 31 slots and
    31 * Hq/Hkv rows per head: several row passes) over prefixes of 0-300 keys;
    every row of the attention output against the oracle."""
    rng = np.random.default_rng(hq * 100 + hkv)
    pool = synth.micro_pool(rng, int(rng.integers(3, 24)), 30, p_neg_inf=0.05)
    N = int(pool["cand_offsets"][-1])
    b = make_micro_batch(pool, max(1, N * 3 // 4), hq=hq, hkv=hkv, p_range=(0, 300),
                         seed=hq + hkv)
    _check_all(b)


def _check_mask_only(b, offset):
    """echo_build_tree_mask on the oracle's selection stored `offset` bytes past a
    16-byte boundary: every output equal to the oracle's."""
    import torch
    import paper_2604_09603_amd as pkg
    cfg = b["cfg"]
    g = oracle.gate(b["cand_offsets"], b["parent"], b["logq"], cfg.budget)
    m = oracle.build_tree_mask(b["cand_offsets"], b["parent"], b["token"], g["selected"],
                               b["root_token"], b["prefix_len"], cfg.budget, cfg.mask_words)
    R, N, B, W = cfg.R, int(b["cand_offsets"][-1]), cfg.budget, cfg.mask_words
    d = torch.device("cuda:0")
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(d)
    raw = torch.zeros(N + 64, dtype=torch.uint8, device=d)
    base = (-raw.data_ptr()) % 16
    sel = raw[base + offset:base + offset + N]
    sel.copy_(dev(g["selected"].astype(np.uint8)))
    assert sel.data_ptr() % 16 == offset % 16
    cap = R + B
    i32 = lambda n: torch.full((n,), -7, dtype=torch.int32, device=d)
    q_offsets, slot_cand, slot_parent, slot_token, pos = i32(R + 1), i32(cap), i32(cap), i32(cap), i32(cap)
    tree_mask = torch.zeros(cap * W, dtype=torch.int32, device=d)
    status = torch.zeros(1, dtype=torch.int32, device=d)
    pkg.echo_build_tree_mask(dev(b["cand_offsets"]), dev(b["parent"]), dev(b["token"]), sel,
                             dev(b["root_token"]), dev(b["prefix_len"]), R, N, B, q_offsets,
                             slot_cand, slot_parent, slot_token, pos, tree_mask, W, status=status)
    torch.cuda.synchronize()
    ns = int(m["num_slots"])
    assert np.array_equal(q_offsets.cpu().numpy(), m["q_offsets"])
    assert np.array_equal(slot_cand.cpu().numpy()[:ns], m["slot_cand"][:ns])
    assert np.array_equal(slot_parent.cpu().numpy()[:ns], m["slot_parent"][:ns])
    assert np.array_equal(slot_token.cpu().numpy()[:ns], m["slot_token"][:ns])
    assert np.array_equal(pos.cpu().numpy()[:ns], m["position_ids"][:ns])
    tm = tree_mask.cpu().numpy().view(np.uint32).reshape(cap, W)
    assert np.array_equal(tm[:ns], np.asarray(m["tree_mask"]).reshape(-1, W)[:ns].view(np.uint32))
    assert int(status.cpu()[0]) == int(m["status"])


@pytest.mark.parametrize("name,offset", [("tiny", 1), ("tiny", 3), ("l8b", 1), ("l8b", 2)])
def test_mask_from_unaligned_selection(name, offset):
    """The packed mask of a selection array that starts off a 16-byte boundary (the
    byte-wise load path) and, for tiny, ends inside a 16-byte chunk."""
    b = synth.make_batch(name, 3)
    print(f"[edges] unaligned selection {name} offset {offset} N={int(b['cand_offsets'][-1])}",
          flush=True)
    _check_mask_only(b, offset)


@pytest.mark.parametrize("offset", [0, 5])
def test_mask_over_several_compaction_rounds(offset):
    """More candidates than one round of the mask kernel's compaction reads
    (1024 threads x 128 flags = 131072): 512 requests of 8 + 6 x 64 = 392 draft
    nodes (N = 200704, two rounds, the second ending inside a wave's range),
    budget 4096 spread over the whole pool; aligned and unaligned flags."""
    cfg = synth.Config("rounds", 512, 7, 8, 3.0, 1000, 4096, 1, 1, 128, 0, 0, ("const", 0.5))
    b = synth.make_batch(cfg, 11, attention=False)
    b["prefix_len"] = np.random.default_rng(12).integers(0, 5000, 512).astype(np.int32)
    N = int(b["cand_offsets"][-1])
    assert N > 131072
    print(f"[edges] multi-round compaction N={N} offset {offset}", flush=True)
    _check_mask_only(b, offset)
