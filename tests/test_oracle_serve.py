"""Pins for the oracle's serving-step pieces: target argmax, acceptance from
logits, paged-cache attention and the KV commit of the accepted path."""
import numpy as np
import pytest

import oracle
from oracle import status as st
import synth
from synth.batch import f32_to_bf16_bits


def _bf(x):
    return f32_to_bf16_bits(np.asarray(x, np.float32))


def test_argmax_closed_forms():
    nan, inf = float("nan"), float("inf")
    rows = [
        ([1.0, 3.0, 3.0, 2.0], 1),          # tie: the smaller id
        ([-0.0, 0.0, -1.0], 0),             # -0 == +0: the smaller id
        ([nan, -5.0, nan, -5.0], 1),        # NaN never wins over a number
        ([nan, nan, nan], 0),               # NaN only: 0
        ([-inf, -inf, nan], 0),
        ([nan, -inf], 1),
        ([2.0, inf, inf], 1),
        ([0.5], 0),
    ]
    for r, want in rows:
        assert oracle.target_argmax(_bf(r)[None, :], 1).tolist() == [want], r


@pytest.mark.parametrize("seed", range(5))
def test_argmax_against_sorting(seed):
    """The argmax is the head of the order (value descending, id ascending)."""
    rng = np.random.default_rng(seed)
    V = 300
    vals = rng.choice(np.array([-2.0, -1.0, 0.0, 0.5, 1.5, -np.inf], np.float32), (20, V))
    logits = _bf(vals)
    got = oracle.target_argmax(logits, 20)
    for s in range(20):
        order = sorted(range(V), key=lambda v: (-float(vals[s, v]), v))
        assert got[s] == order[0]


def test_accept_from_logits_matches_accept_with_targets():
    rng = np.random.default_rng(3)
    b = synth.micro_pool(rng, 4, 10)
    g = oracle.gate(b["cand_offsets"], b["parent"], b["logq"], 12)
    m = oracle.build_tree_mask(b["cand_offsets"], b["parent"], b["token"], g["selected"],
                               b["root_token"], b["prefix_len"], 12, 1)
    nq = m["num_slots"]
    V = 7
    tgt = rng.integers(0, V, nq).astype(np.int32)
    logits = _bf(rng.normal(size=(nq, V)).astype(np.float32) - 10.0)
    logits[np.arange(nq), tgt] = _bf([3.0])[0]         # one clear winner per row
    a = oracle.accept_from_logits(m["q_offsets"], m["slot_parent"], m["slot_token"], logits, 16)
    ref = oracle.accept(m["q_offsets"], m["slot_parent"], m["slot_token"], tgt, 16)
    assert np.array_equal(a["target_token"], tgt)
    for k in ("accept_len", "accept_slots", "bonus_token"):
        assert np.array_equal(a[k], ref[k])


def _paged_case(seed, page_size=4, R=3, hkv=2, hq=4):
    """A small batch with its prefixes laid out both contiguously and in
    shuffled pages."""
    rng = np.random.default_rng(seed)
    P = rng.integers(0, 11, R).astype(np.int32)
    D = 128
    kvo = np.zeros(R + 1, np.int64)
    kvo[1:] = np.cumsum(P)
    T = int(kvo[-1])
    kc = _bf(rng.normal(size=(T, hkv, D)))
    vc = _bf(rng.normal(size=(T, hkv, D)))
    npg = [int((p + page_size - 1) // page_size) for p in P]
    maxp = max(npg) + 2
    total = sum(npg) + 3
    perm = rng.permutation(total)
    bt = np.full((R, maxp), -1, np.int32)
    kp = _bf(rng.normal(size=(total, page_size, hkv, D)))   # junk outside the prefixes
    vp = _bf(rng.normal(size=(total, page_size, hkv, D)))
    k = 0
    for r in range(R):
        for e in range(npg[r]):
            page = int(perm[k]); k += 1
            bt[r, e] = page
            for j in range(page_size):
                pos = e * page_size + j
                if pos < P[r]:
                    kp[page, j] = kc[kvo[r] + pos]
                    vp[page, j] = vc[kvo[r] + pos]
    n = rng.integers(1, 4, R)
    qo = np.zeros(R + 1, np.int32)
    qo[1:] = np.cumsum(n)
    cap = int(qo[-1])
    W = 1
    mask = np.zeros((cap, W), np.uint32)
    par = np.full(cap, -1, np.int32)
    for r in range(R):
        for s in range(int(n[r])):
            bits = 1 << s
            if s > 0:
                par[qo[r] + s] = int(rng.integers(0, s))
                bits |= int(mask[qo[r] + par[qo[r] + s], 0])
            mask[qo[r] + s, 0] = bits
    q = _bf(rng.normal(size=(cap, hq, D)))
    kn = _bf(rng.normal(size=(cap, hkv, D)))
    vn = _bf(rng.normal(size=(cap, hkv, D)))
    return dict(P=P, kvo=kvo, kc=kc, vc=vc, kp=kp, vp=vp, bt=bt, qo=qo, mask=mask, q=q, kn=kn,
                vn=vn, hq=hq, hkv=hkv, page_size=page_size, par=par, n=n)


@pytest.mark.parametrize("seed", range(4))
def test_paged_attention_equals_contiguous(seed):
    """Shuffled pages read through the block table give the contiguous result."""
    c = _paged_case(seed)
    scale = np.float32(1 / np.sqrt(128))
    ref, rl, s0 = oracle.tree_verify_attn(c["q"], c["kn"], c["vn"], c["kc"], c["vc"], c["kvo"],
                                          c["qo"], c["mask"], c["hq"], c["hkv"], scale)
    got, gl, s1 = oracle.tree_verify_attn_paged(c["q"], c["kn"], c["vn"], c["kp"], c["vp"],
                                                c["bt"], c["P"], c["page_size"], c["qo"],
                                                c["mask"], c["hq"], c["hkv"], scale)
    assert s0 == s1 == 0
    assert np.array_equal(ref, got) and np.array_equal(rl, gl)


def test_paged_attention_missing_page():
    c = _paged_case(7)
    r = int(np.argmax(c["P"]))
    c["bt"][r, 0] = -1
    scale = np.float32(1 / np.sqrt(128))
    out, lse, s = oracle.tree_verify_attn_paged(c["q"], c["kn"], c["vn"], c["kp"], c["vp"],
                                                c["bt"], c["P"], c["page_size"], c["qo"],
                                                c["mask"], c["hq"], c["hkv"], scale)
    assert s == st.BAD_OFFSETS
    rows = range(int(c["qo"][r]), int(c["qo"][r + 1]))
    assert np.all(np.isnan(out[list(rows)]))


def test_commit_appends_root_and_accepted_path():
    """Hand-built: request 0 accepts 2 slots, request 1 none, request 2 has no slot."""
    page_size, hkv, D = 4, 1, 128
    kp = np.zeros((6, page_size, hkv, D), np.uint16)
    vp = np.zeros_like(kp)
    bt = np.array([[2, 5, -1], [0, -1, -1], [1, -1, -1]], np.int32)
    P = np.array([3, 1, 2], np.int32)
    qo = np.array([0, 4, 6, 6], np.int32)
    kn = np.arange(6 * hkv * D, dtype=np.uint16).reshape(6, hkv, D)
    vn = kn + np.uint16(1000)
    acc_len = np.array([2, 0, 0], np.int32)
    acc_slots = np.array([[2, 3, -1], [-1] * 3, [-1] * 3], np.int32)
    kp2, vp2, P2, s = oracle.commit_kv(qo, acc_len, acc_slots, kn, vn, kp, vp, bt, P, page_size)
    assert s == 0
    assert P2.tolist() == [6, 2, 2]
    # request 0: positions 3 (root slot 0), 4 (slot 2), 5 (slot 3): page 2 row 3, page 5 rows 0-1
    assert np.array_equal(kp2[2, 3], kn[0]) and np.array_equal(kp2[5, 0], kn[2])
    assert np.array_equal(kp2[5, 1], kn[3]) and np.array_equal(vp2[5, 1], vn[3])
    # request 1: its root (slot 4) at position 1 of page 0
    assert np.array_equal(kp2[0, 1], kn[4])
    # nothing else moved
    changed = {(2, 3), (5, 0), (5, 1), (0, 1)}
    for pg in range(6):
        for row in range(page_size):
            if (pg, row) not in changed:
                assert not kp2[pg, row].any() and not vp2[pg, row].any()


def test_commit_missing_page_leaves_the_request():
    page_size, hkv, D = 2, 1, 128
    kp = np.zeros((3, page_size, hkv, D), np.uint16)
    bt = np.array([[0, -1]], np.int32)                    # position 2 has no page
    kn = np.ones((3, hkv, D), np.uint16)
    kp2, vp2, P2, s = oracle.commit_kv(np.array([0, 3], np.int32), np.array([2], np.int32),
                                       np.array([[1, 2]], np.int32), kn, kn, kp, kp.copy(), bt,
                                       np.array([1], np.int32), page_size)
    assert s == st.BAD_OFFSETS and P2.tolist() == [1] and not kp2.any()


def test_commit_then_decode_equals_contiguous_history():
    """After a commit, attention of a new root over the paged prefix equals
    attention over the old prefix with the committed rows appended."""
    c = _paged_case(11, page_size=4)
    R = len(c["P"])
    # give every request room for 4 more positions
    extra = 4
    total = c["kp"].shape[0]
    bt = c["bt"].copy()
    kp = np.concatenate([c["kp"], np.zeros((R * 2, 4, c["hkv"], 128), np.uint16)])
    vp = np.concatenate([c["vp"], np.zeros_like(kp[total:])])
    nxt = total
    for r in range(R):
        need = (int(c["P"][r]) + extra + 3) // 4
        for e in range(need):
            if bt[r, e] < 0:
                bt[r, e] = nxt
                nxt += 1
    acc_len = np.array([min(1, int(c["n"][r]) - 1) for r in range(R)], np.int32)
    acc_slots = np.full((R, 16), -1, np.int32)
    for r in range(R):
        if acc_len[r]:
            acc_slots[r, 0] = int(c["qo"][r]) + 1
    kp2, vp2, P2, s = oracle.commit_kv(c["qo"], acc_len, acc_slots, c["kn"], c["vn"], kp, vp, bt,
                                       c["P"], 4)
    assert s == 0
    hist_k, hist_v = [], []
    for r in range(R):
        rows = [int(c["qo"][r])] + [int(x) for x in acc_slots[r, :acc_len[r]]]
        hist_k.append(np.concatenate([c["kc"][c["kvo"][r]:c["kvo"][r + 1]], c["kn"][rows]]))
        hist_v.append(np.concatenate([c["vc"][c["kvo"][r]:c["kvo"][r + 1]], c["vn"][rows]]))
    kvo = np.zeros(R + 1, np.int64)
    kvo[1:] = np.cumsum([len(h) for h in hist_k])
    rng = np.random.default_rng(5)
    q1 = _bf(rng.normal(size=(R, c["hq"], 128)))
    k1 = _bf(rng.normal(size=(R, c["hkv"], 128)))
    qo1 = np.arange(R + 1, dtype=np.int32)
    mask1 = np.ones((R, 1), np.uint32)
    scale = np.float32(1 / np.sqrt(128))
    ref = oracle.tree_verify_attn(q1, k1, k1, np.concatenate(hist_k), np.concatenate(hist_v), kvo,
                                  qo1, mask1, c["hq"], c["hkv"], scale)
    got = oracle.tree_verify_attn_paged(q1, k1, k1, kp2, vp2, bt, P2, 4, qo1, mask1, c["hq"],
                                        c["hkv"], scale)
    assert np.array_equal(ref[0], got[0])
