"""Pins for the float64 oracle attention: dense brute force, causal reduction, closed forms."""
import math

import numpy as np
import pytest
import torch

import oracle
import synth
from tests import bruteforce as bf


def _bf16(rng, *shape, scale=1.0):
    return synth.f32_to_bf16_bits((rng.standard_normal(shape) * scale).astype(np.float32))


def _f64(bits):
    return synth.bf16_bits_to_f32(bits).astype(np.float64)


def _inputs(rng, pool, budget, hq, hkv, D, P):
    offs = pool["cand_offsets"]
    R = len(offs) - 1
    g = oracle.gate(offs, pool["parent"], pool["logq"], budget)
    W = (budget + 1 + 31) // 32
    m = oracle.build_tree_mask(offs, pool["parent"], pool["token"], g["selected"],
                               pool["root_token"], np.asarray(P, np.int32), budget, W)
    cap = R + budget
    kvo = np.zeros(R + 1, np.int64)
    kvo[1:] = np.cumsum(P)
    T = int(kvo[-1])
    return dict(q=_bf16(rng, cap, hq, D), k_new=_bf16(rng, cap, hkv, D), v_new=_bf16(rng, cap, hkv, D),
                k_cache=_bf16(rng, T, hkv, D), v_cache=_bf16(rng, T, hkv, D), kv_offsets=kvo,
                q_offsets=m["q_offsets"], tree_mask=m["tree_mask"], slot_parent=m["slot_parent"],
                hq=hq, hkv=hkv, sm_scale=np.float32(1 / math.sqrt(D)))


def _run(x, rows=None):
    return oracle.tree_verify_attn(x["q"], x["k_new"], x["v_new"], x["k_cache"], x["v_cache"],
                                   x["kv_offsets"], x["q_offsets"], x["tree_mask"], x["hq"],
                                   x["hkv"], x["sm_scale"], rows=rows)


def _vis_from_parents(x):
    """Global slots each slot sees, from the dense closure of slot_parent (not the bits)."""
    qo = x["q_offsets"]
    vis = {}
    for r in range(len(qo) - 1):
        s0, s1 = int(qo[r]), int(qo[r + 1])
        A = bf.transitive_closure(x["slot_parent"][s0:s1].tolist())
        for j in range(s1 - s0):
            vis[s0 + j] = [s0 + i for i in np.nonzero(A[j])[0]]
    return vis


@pytest.mark.parametrize("seed", range(12))
def test_attn_matches_dense_masked_softmax(seed):
    rng = np.random.default_rng(seed)
    pool = synth.micro_pool(rng, 3, 6)
    hq, hkv = [(4, 2), (2, 2), (6, 1)][seed % 3]
    P = rng.integers(0, 6, size=3)
    x = _inputs(rng, pool, int(rng.integers(0, 10)), hq, hkv, 16, P)
    out, lse, status = _run(x)
    assert status == 0
    ref, ref_lse = bf.dense_attention(x["q"], x["k_new"], x["v_new"], x["k_cache"], x["v_cache"],
                                      x["kv_offsets"], x["q_offsets"], _vis_from_parents(x), hq, hkv,
                                      x["sm_scale"])
    np.testing.assert_allclose(out, ref, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(lse, ref_lse, rtol=1e-12, atol=1e-12)


def test_single_path_tree_is_causal_attention():
    """A chain-shaped selected tree reduces to ordinary causal attention over prefix + chain."""
    rng = np.random.default_rng(5)
    n, P, hq, hkv, D = 5, 9, 4, 2, 128
    pool = dict(cand_offsets=np.array([0, n], np.int32),
                parent=np.array([-1] + list(range(n - 1)), np.int32),
                token=np.arange(n, dtype=np.int32), logq=np.full(n, -0.5, np.float32),
                root_token=np.array([1], np.int32))
    x = _inputs(rng, pool, n, hq, hkv, D, np.array([P]))
    out, lse, _ = _run(x)
    L = n + 1
    keys = np.concatenate([_f64(x["k_cache"][:P]), _f64(x["k_new"][:L])], axis=0)  # [P+L, Hkv, D]
    vals = np.concatenate([_f64(x["v_cache"][:P]), _f64(x["v_new"][:L])], axis=0)
    causal = torch.ones(L, P + L, dtype=torch.bool).tril(diagonal=P)             # bottom-right causal
    G = hq // hkv
    for h in range(hq):
        qh = torch.from_numpy(_f64(x["q"][:L, h]))[None, None]
        kh = torch.from_numpy(keys[:, h // G])[None, None]
        vh = torch.from_numpy(vals[:, h // G])[None, None]
        ref = torch.nn.functional.scaled_dot_product_attention(
            qh, kh, vh, attn_mask=causal, scale=float(x["sm_scale"]))[0, 0].numpy()
        np.testing.assert_allclose(out[:L, h], ref, rtol=1e-10, atol=1e-12)


def test_budget_zero_is_decode_attention():
    """B = 0: each root attends to its prefix plus itself: plain decode attention."""
    rng = np.random.default_rng(9)
    pool = synth.micro_pool(rng, 3, 4)
    P = np.array([7, 1, 12])
    x = _inputs(rng, pool, 0, 4, 1, 64, P)
    out, lse, _ = _run(x)
    for r in range(3):
        k0, k1 = int(x["kv_offsets"][r]), int(x["kv_offsets"][r + 1])
        keys = np.concatenate([_f64(x["k_cache"][k0:k1, 0]), _f64(x["k_new"][r:r + 1, 0])])
        vals = np.concatenate([_f64(x["v_cache"][k0:k1, 0]), _f64(x["v_new"][r:r + 1, 0])])
        for h in range(4):
            ref = torch.nn.functional.scaled_dot_product_attention(
                torch.from_numpy(_f64(x["q"][r, h]))[None, None, None],
                torch.from_numpy(keys)[None, None], torch.from_numpy(vals)[None, None],
                scale=float(x["sm_scale"]))[0, 0, 0].numpy()
            np.testing.assert_allclose(out[r, h], ref, rtol=1e-10, atol=1e-12)


def test_closed_forms():
    rng = np.random.default_rng(11)
    pool = synth.micro_pool(rng, 3, 6, p_neg_inf=0.0)
    P = np.array([3, 0, 5])
    x = _inputs(rng, pool, 8, 4, 2, 32, P)
    vis = _vis_from_parents(x)
    # constant V  ->  O = V
    c = _bf16(rng, 1, 2, 32)
    x1 = dict(x, v_new=np.broadcast_to(c, x["v_new"].shape).copy(),
              v_cache=np.broadcast_to(c, x["v_cache"].shape).copy())
    out, lse, _ = _run(x1)
    for h in range(4):
        np.testing.assert_allclose(out[:, h], np.broadcast_to(_f64(c[0, h // 2]), out[:, h].shape),
                                   rtol=1e-13, atol=1e-13)
    # Q = 0  ->  O = mean of the visible V, LSE = ln(#visible)
    x2 = dict(x, q=np.zeros_like(x["q"]))
    out, lse, _ = _run(x2)
    qo = x["q_offsets"]
    for r in range(3):
        k0, k1 = int(x["kv_offsets"][r]), int(x["kv_offsets"][r + 1])
        for s in range(int(qo[r]), int(qo[r + 1])):
            for h in range(4):
                rows = [_f64(x["v_cache"][t, h // 2]) for t in range(k0, k1)]
                rows += [_f64(x["v_new"][j, h // 2]) for j in vis[s]]
                np.testing.assert_allclose(out[s, h], np.mean(rows, axis=0), rtol=1e-12, atol=1e-14)
                assert abs(lse[s, h] - math.log(len(rows))) < 1e-13


def test_row_without_keys():
    """No prefix and no mask bit: output 0 and LSE -inf."""
    rng = np.random.default_rng(2)
    x = dict(q=_bf16(rng, 2, 2, 8), k_new=_bf16(rng, 2, 1, 8), v_new=_bf16(rng, 2, 1, 8),
             k_cache=_bf16(rng, 0, 1, 8), v_cache=_bf16(rng, 0, 1, 8),
             kv_offsets=np.array([0, 0], np.int64), q_offsets=np.array([0, 2], np.int32),
             tree_mask=np.array([[1], [0]], np.uint32), hq=2, hkv=1, sm_scale=np.float32(0.5))
    out, lse, _ = _run(x)
    assert np.all(out[1] == 0) and np.all(np.isneginf(lse[1]))
    assert np.all(np.isfinite(out[0]))


def test_row_subset_matches_full():
    rng = np.random.default_rng(4)
    pool = synth.micro_pool(rng, 3, 6)
    x = _inputs(rng, pool, 6, 4, 2, 16, np.array([4, 2, 3]))
    full, full_lse, _ = _run(x)
    rows = [0, 2, int(x["q_offsets"][-1]) - 1]
    part, part_lse, _ = _run(x, rows=rows)
    np.testing.assert_array_equal(part[rows], full[rows])
    np.testing.assert_array_equal(part_lse[rows], full_lse[rows])
