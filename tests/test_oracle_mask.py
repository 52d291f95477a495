"""Pins for the oracle flatten & pack (Fig. 3 stage 3): slots, positions, ancestor bitmasks."""
import json
import os

import numpy as np
import pytest

import oracle
from oracle import status as st
import synth
from tests import bruteforce as bf

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _check_against_dense(pool, sel, budget, res):
    offs, parent = pool["cand_offsets"], pool["parent"]
    R = len(offs) - 1
    qo = res["q_offsets"]
    assert qo[0] == 0
    for r in range(R):
        lo, hi = int(offs[r]), int(offs[r + 1])
        nodes = [g for g in range(lo, hi) if sel[g]]
        s0, s1 = int(qo[r]), int(qo[r + 1])
        assert s1 - s0 == 1 + len(nodes)
        # slot order: root, then selected candidates in ascending index
        assert res["slot_cand"][s0] == -1
        assert res["slot_cand"][s0 + 1:s1].tolist() == nodes
        assert res["slot_token"][s0] == pool["root_token"][r]
        assert res["slot_token"][s0 + 1:s1].tolist() == [int(pool["token"][g]) for g in nodes]
        n = s1 - s0
        A = bf.transitive_closure(res["slot_parent"][s0:s1].tolist())
        for j in range(n):
            bits = bf.unpack_mask(res["tree_mask"][s0 + j], res["tree_mask"].shape[1] * 32)
            assert np.array_equal(bits[:n], A[j]), (r, j)
            assert not bits[n:].any()
            d = int(bits.sum()) - 1
            # depth from the candidate tree itself (closed selections)
            cand_depth = 0 if j == 0 else len(bf.root_path(offs, parent, int(res["slot_cand"][s0 + j])))
            assert d == cand_depth
            assert res["position_ids"][s0 + j] - pool["prefix_len"][r] == d
        # rows are lower-triangular in local index: ancestors come first
        assert not np.triu(A, 1).any()


@pytest.mark.parametrize("seed", range(40))
def test_mask_matches_dense_closure(seed):
    pool = synth.micro_pool(np.random.default_rng(100 + seed), 4, 10)
    offs = pool["cand_offsets"]
    N = int(offs[-1])
    for budget in sorted({0, 1, 5, N}):
        g = oracle.gate(offs, pool["parent"], pool["logq"], budget)
        W = (budget + 1 + 31) // 32
        res = oracle.build_tree_mask(offs, pool["parent"], pool["token"], g["selected"],
                                     pool["root_token"], pool["prefix_len"], budget, W)
        assert res["status"] == 0
        _check_against_dense(pool, g["selected"], budget, res)


def test_mask_golden_example():
    """Hand-drawn two-request example with the expected layout written out by hand."""
    with open(os.path.join(GOLDEN, "mask_example.json")) as f:
        c = json.load(f)
    res = oracle.build_tree_mask(np.array(c["cand_offsets"]), np.array(c["parent"], np.int32),
                                 np.array(c["token"], np.int32), np.array(c["selected"], np.uint8),
                                 np.array(c["root_token"], np.int32), np.array(c["prefix_len"], np.int32),
                                 c["budget"], c["mask_words"])
    nq = res["num_slots"]
    for key in ["q_offsets", "slot_cand", "slot_parent", "slot_token", "position_ids"]:
        assert res[key][:len(c[key])].tolist() == c[key], key
    assert res["tree_mask"][:nq, 0].tolist() == c["tree_mask_word0"]
    assert res["status"] == 0


def test_mask_many_words():
    """A request with more than 32 slots spreads its bitmask over several words."""
    n = 70
    offs = np.array([0, n], np.int32)
    parent = np.array([-1] + list(range(n - 1)), np.int32)   # a chain: node k's parent is k-1
    sel = np.ones(n, np.uint8)
    res = oracle.build_tree_mask(offs, parent, np.arange(n, dtype=np.int32), sel,
                                 np.array([7], np.int32), np.array([3], np.int32), n, 3)
    for j in range(n + 1):
        bits = bf.unpack_mask(res["tree_mask"][j], 96)
        assert bits[:j + 1].all() and not bits[j + 1:].any()
        assert res["position_ids"][j] == 3 + j


def test_mask_status_rules():
    offs = np.array([0, 4], np.int32)
    parent = np.array([-1, 0, 1, 9], np.int32)
    tok = np.arange(4, dtype=np.int32)
    # node 2 selected without its parent 1: attached to node 0 (NOT_CLOSED); node 3 has a bad parent
    sel = np.array([1, 0, 1, 1], np.uint8)
    res = oracle.build_tree_mask(offs, parent, tok, sel, np.array([5], np.int32),
                                 np.array([10], np.int32), 3, 1)
    assert res["status"] == st.NOT_CLOSED | st.BAD_PARENT
    assert res["slot_parent"][:4].tolist() == [-1, 0, 1, 0]
    assert res["position_ids"][:4].tolist() == [10, 11, 12, 11]
    # more selected nodes than the budget: only the first B packed
    res = oracle.build_tree_mask(offs, parent, tok, np.ones(4, np.uint8), np.array([5], np.int32),
                                 np.array([10], np.int32), 2, 1)
    assert res["status"] & st.OVER_CAPACITY
    assert res["slot_cand"][:3].tolist() == [-1, 0, 1]
    with pytest.raises(ValueError):
        oracle.build_tree_mask(offs, parent, tok, sel, np.array([5], np.int32),
                               np.array([10], np.int32), 40, 1)


@pytest.mark.parametrize("name", ["tiny", "l8b"])
def test_mask_on_presets(name):
    b = synth.make_batch(name, 1, attention=False)
    cfg = b["cfg"]
    b["prefix_len"] = np.full(cfg.R, 100, np.int32)
    g = oracle.gate(b["cand_offsets"], b["parent"], b["logq"], cfg.budget)
    res = oracle.build_tree_mask(b["cand_offsets"], b["parent"], b["token"], g["selected"],
                                 b["root_token"], b["prefix_len"], cfg.budget, cfg.mask_words)
    assert res["status"] == 0
    assert res["num_slots"] == cfg.R + g["num_selected"]
    _check_against_dense(b, g["selected"], cfg.budget, res)


def test_malformed_csr_packs_roots_only():
    offs = np.array([0, 6, 4, 9], np.int32)          # decreasing: malformed
    N = 9
    selected = np.ones(N, np.uint8)
    m = oracle.build_tree_mask(offs, np.full(N, -1, np.int32), np.arange(N, dtype=np.int32),
                               selected, np.array([7, 8, 9], np.int32),
                               np.array([3, 0, 5], np.int32), budget=4, mask_words=1)
    assert m["status"] & oracle.status.BAD_OFFSETS
    assert m["q_offsets"].tolist() == [0, 1, 2, 3]
    assert m["slot_token"][:3].tolist() == [7, 8, 9]
    assert m["position_ids"][:3].tolist() == [3, 0, 5]
    assert m["tree_mask"][:3, 0].tolist() == [1, 1, 1]
