"""Pins for the oracle greedy acceptance: path enumeration and closed forms."""
import json
import os

import numpy as np
import pytest

import oracle
from oracle import status as st
import synth
from tests import bruteforce as bf

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


@pytest.mark.parametrize("seed", range(40))
def test_accept_matches_path_enumeration(seed):
    rng = np.random.default_rng(300 + seed)
    pool = synth.micro_pool(rng, 4, 9, vocab=3)       # tiny vocab: many matches, duplicate siblings
    offs = pool["cand_offsets"]
    N = int(offs[-1])
    budget = int(rng.integers(0, N + 1))
    g = oracle.gate(offs, pool["parent"], pool["logq"], budget)
    m = oracle.build_tree_mask(offs, pool["parent"], pool["token"], g["selected"], pool["root_token"],
                               pool["prefix_len"], budget, (budget + 32) // 32)
    nq = m["num_slots"]
    target = rng.integers(0, 3, size=nq).astype(np.int32)
    max_depth = int(rng.integers(1, 17))
    res = oracle.accept(m["q_offsets"], m["slot_parent"], m["slot_token"], target, max_depth)
    assert res["status"] == 0
    qo = m["q_offsets"]
    for r in range(len(qo) - 1):
        s0, s1 = int(qo[r]), int(qo[r + 1])
        d, end, path = bf.brute_accept(s1 - s0, m["slot_parent"][s0:s1].tolist(),
                                       m["slot_token"][s0:s1].tolist(), target[s0:s1].tolist(),
                                       max_depth)
        assert res["accept_len"][r] == d
        assert res["accept_slots"][r, :d].tolist() == [s0 + j for j in path]
        assert np.all(res["accept_slots"][r, d:] == -1)
        assert res["bonus_token"][r] == target[s0 + end]


def test_accept_closed_forms():
    # a chain root -> 1 -> 2 -> 3 where the target always predicts the next draft token
    qo = np.array([0, 4], np.int32)
    sp = np.array([-1, 0, 1, 2], np.int32)
    tok = np.array([50, 7, 8, 9], np.int32)
    tgt = np.array([7, 8, 9, 42], np.int32)
    res = oracle.accept(qo, sp, tok, tgt, 16)
    assert res["accept_len"].tolist() == [3]
    assert res["accept_slots"][0, :4].tolist() == [1, 2, 3, -1]
    assert res["bonus_token"].tolist() == [42]
    # max_depth caps the path
    res = oracle.accept(qo, sp, tok, tgt, 2)
    assert res["accept_len"].tolist() == [2] and res["bonus_token"].tolist() == [9]
    # nothing matches: length 0 and the bonus is the target after the root
    res = oracle.accept(qo, sp, tok, np.array([1, 1, 1, 1], np.int32), 16)
    assert res["accept_len"].tolist() == [0] and res["bonus_token"].tolist() == [1]
    assert np.all(res["accept_slots"] == -1)


def test_accept_golden_example():
    with open(os.path.join(GOLDEN, "accept_example.json")) as f:
        c = json.load(f)
    res = oracle.accept(np.array(c["q_offsets"]), np.array(c["slot_parent"]), np.array(c["slot_token"]),
                        np.array(c["target_token"]), c["max_depth"])
    assert res["accept_len"].tolist() == c["accept_len"]
    assert res["accept_slots"].tolist() == c["accept_slots"]
    assert res["bonus_token"].tolist() == c["bonus_token"]
    assert res["status"] == 0


def test_accept_status_and_empty():
    qo = np.array([0, 3, 3], np.int32)                 # request 1 has no slots
    sp = np.array([-1, 2, 0], np.int32)                # slot 1 points forward: unacceptable
    tok = np.array([0, 5, 6], np.int32)
    tgt = np.array([5, 0, 0], np.int32)
    res = oracle.accept(qo, sp, tok, tgt, 4)
    assert res["status"] == st.BAD_SLOT_PARENT
    assert res["accept_len"].tolist() == [0, 0]
    assert res["bonus_token"].tolist() == [5, -1]


@pytest.mark.parametrize("name", ["tiny", "l8b"])
def test_accept_on_presets_follows_top1_chain(name):
    """With the stand-in target, an accepted path only ever follows top-1 children."""
    b = synth.make_batch(name, 2, attention=False)
    cfg = b["cfg"]
    P = np.full(cfg.R, 10, np.int32)
    g = oracle.gate(b["cand_offsets"], b["parent"], b["logq"], cfg.budget)
    m = oracle.build_tree_mask(b["cand_offsets"], b["parent"], b["token"], g["selected"],
                               b["root_token"], P, cfg.budget, cfg.mask_words)
    tgt = synth.target_for_slots(b, m["q_offsets"], m["slot_cand"])
    res = oracle.accept(m["q_offsets"], m["slot_parent"], m["slot_token"], tgt, 16)
    assert res["status"] == 0
    assert res["accept_len"].max() <= cfg.depth
    assert (res["accept_len"] > 0).any()
