"""The seeded generator: reproducibility and the structural invariants of its trees."""
import hashlib

import numpy as np
import pytest

import synth


def _digest(b):
    h = hashlib.sha256()
    for k in sorted(b):
        v = b[k]
        if isinstance(v, np.ndarray):
            h.update(k.encode()); h.update(np.ascontiguousarray(v).tobytes())
    return h.hexdigest()


def test_same_seed_same_bytes():
    a = synth.make_batch("tiny", 3)
    b = synth.make_batch("tiny", 3)
    c = synth.make_batch("tiny", 4)
    assert _digest(a) == _digest(b) != _digest(c)


@pytest.mark.parametrize("name", ["tiny", "l8b"])
def test_tree_invariants(name):
    b = synth.make_batch(name, 0, attention=(name == "tiny"))
    cfg = b["cfg"]
    offs = b["cand_offsets"]
    assert len(offs) == cfg.R + 1
    assert np.all(np.diff(offs) == cfg.nodes_per_request)
    for r in range(cfg.R):
        lo, hi = offs[r], offs[r + 1]
        par = b["parent"][lo:hi]
        assert np.all(par < np.arange(hi - lo)) and np.all(par >= -1)
        depth = np.zeros(hi - lo, int)
        for n in range(hi - lo):
            depth[n] = 1 if par[n] < 0 else depth[par[n]] + 1
        assert depth.max() == cfg.depth
        assert np.bincount(depth)[1:].tolist() == [cfg.branch] + [cfg.branch ** 2] * (cfg.depth - 1)
        # siblings carry distinct tokens, in descending draft probability
        for p in np.unique(par):
            kids = np.nonzero(par == p)[0]
            assert len(set(b["token"][lo + kids])) == len(kids)
            assert np.all(np.diff(b["logq"][lo + kids]) <= 0)
    assert np.all(b["logq"] <= 0) and np.all(np.isfinite(b["logq"]))
    assert np.all((b["token"] >= 0) & (b["token"] < cfg.vocab))
    if "prefix_len" in b:
        assert np.all((b["prefix_len"] >= cfg.p_lo) & (b["prefix_len"] <= cfg.p_hi))
        assert b["k_cache"].shape == (int(b["kv_offsets"][-1]), cfg.hkv, cfg.head_dim)
        assert b["q"].shape == (cfg.capacity, cfg.hq, cfg.head_dim)


def test_bf16_rounding_is_nearest_even():
    # bf16 keeps 8 significant bits: the spacing just above 1.0 is 2^-7
    x = np.array([1.0 + 2 ** -7, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -2.5, 1.0 + 3 * 2 ** -9], np.float32)
    back = synth.bf16_bits_to_f32(synth.f32_to_bf16_bits(x))
    # exact; tie -> even (1.0); tie -> even (1+2^-6); exact; nearer to 1+2^-7
    assert back.tolist() == [1.0 + 2 ** -7, 1.0, 1.0 + 2 ** -6, -2.5, 1.0 + 2 ** -7]
