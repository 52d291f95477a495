"""Oracle post-verification step of a serving loop: the target argmax that
acceptance consumes, the KV-cache commit of the accepted path, and
verification attention over a paged KV cache.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The paper runs greedy decoding (Section 2, "Standard SD"; Section 5.1): the
target's token after each verified slot is the argmax of its logits, and a
draft token is accepted when it equals the argmax after its parent.  After
acceptance the accepted path's keys and values join the request's KV cache
(the paper leaves the cache's layout to the serving engine; a block table of
fixed-size pages is the common one).  Conventions of this library:

* argmax over the vocabulary of the bfloat16 logits, compared as floats
  (-0 == +0); NaN never wins over a number; ties go to the smaller token id;
* a paged cache stores position p of request r in page
  block_table[r][p // page_size] at row p % page_size, each row holding all
  KV heads;
* the commit appends the root slot (position P_r) and the accepted slots
  (positions P_r + 1 .. P_r + accept_len) of each request and advances P_r by
  1 + accept_len.  A request whose block table lacks a page it needs is left
  unchanged (status BAD_OFFSETS).
"""
import numpy as np

from . import status as st
from .accept import accept
from .attn import tree_verify_attn


def _bf16_to_f32(bits):
    b = np.asarray(bits, np.uint16).astype(np.uint32) << 16
    return b.view(np.float32)


def target_argmax(logits, rows):
    """Greedy target token of each of the first ``rows`` rows of bf16 ``logits``
    [cap, V]: the smallest index of the largest value, NaN ignored (a row of
    NaN only gives 0)."""
    out = np.zeros(rows, np.int32)
    for s in range(rows):
        x = _bf16_to_f32(logits[s])
        idx = np.flatnonzero(~np.isnan(x))
        if idx.size:
            out[s] = idx[int(np.argmax(x[idx]))]   # np.argmax keeps the first maximum
    return out


def accept_from_logits(q_offsets, slot_parent, slot_token, logits, max_depth):
    """Greedy acceptance with the target argmax taken from the logits."""
    nq = int(np.asarray(q_offsets)[-1])
    tgt = target_argmax(logits, nq)
    res = accept(q_offsets, slot_parent, slot_token, tgt, max_depth)
    res["target_token"] = tgt
    return res


def paged_rows(pages, block_table, r, length, page_size):
    """Rows 0 .. length-1 of request r from a paged cache, or None if a page is
    missing or out of range."""
    rows = []
    for p in range(length):
        e = p // page_size
        if e >= block_table.shape[1]:
            return None
        page = int(block_table[r, e])
        if page < 0 or page >= pages.shape[0]:
            return None
        rows.append(pages[page, p % page_size])
    return np.stack(rows) if rows else pages[:0, 0]


def tree_verify_attn_paged(q, k_new, v_new, k_pages, v_pages, block_table, prefix_len,
                           page_size, q_offsets, tree_mask, hq, hkv, sm_scale, rows=None):
    """Verification attention with each request's prefix read through its block
    table: the prefixes are gathered into one token-major cache and the
    contiguous oracle runs on it.  A request with a missing page gets no
    output (its rows stay NaN) and BAD_OFFSETS."""
    R = len(q_offsets) - 1
    status = 0
    parts, lens = [], []
    skip = set()
    for r in range(R):
        P = int(prefix_len[r])
        got = None if P < 0 else paged_rows(k_pages, block_table, r, P, page_size)
        if got is None:
            status |= st.BAD_OFFSETS
            skip.add(r)
            parts.append((k_pages[:0, 0], v_pages[:0, 0]))
            lens.append(0)
            continue
        parts.append((got, paged_rows(v_pages, block_table, r, P, page_size)))
        lens.append(P)
    kv_offsets = np.zeros(R + 1, np.int64)
    kv_offsets[1:] = np.cumsum(lens)
    k_cache = np.concatenate([p[0] for p in parts]) if R else k_pages[:0, 0]
    v_cache = np.concatenate([p[1] for p in parts]) if R else v_pages[:0, 0]
    qo = np.asarray(q_offsets, np.int64)
    want = [s for r in range(R) if r not in skip for s in range(int(qo[r]), int(qo[r + 1]))]
    if rows is not None:
        rs = set(int(x) for x in rows)
        want = [s for s in want if s in rs]
    out, lse, st2 = tree_verify_attn(q, k_new, v_new, k_cache, v_cache, kv_offsets, q_offsets,
                                     tree_mask, hq, hkv, sm_scale, rows=want)
    return out, lse, status | st2


def commit_kv(q_offsets, accept_len, accept_slots, k_new, v_new, k_pages, v_pages, block_table,
              prefix_len, page_size):
    """Return (k_pages', v_pages', prefix_len', status) after appending each
    request's root slot and accepted slots at positions P_r, P_r + 1, ..."""
    kp, vp = k_pages.copy(), v_pages.copy()
    plen = np.asarray(prefix_len, np.int32).copy()
    qo = np.asarray(q_offsets, np.int64)
    status = 0
    for r in range(len(qo) - 1):
        if int(qo[r + 1]) <= int(qo[r]):
            continue                      # no slot: nothing verified, nothing to commit
        L = int(accept_len[r])
        slots = [int(qo[r])] + [int(x) for x in accept_slots[r, :L]]
        P = int(plen[r])
        dest = []
        for j in range(len(slots)):
            p = P + j
            e = p // page_size
            page = int(block_table[r, e]) if 0 <= e < block_table.shape[1] else -1
            if page < 0 or page >= kp.shape[0]:
                dest = None
                break
            dest.append((page, p % page_size))
        if dest is None:
            status |= st.BAD_OFFSETS
            continue
        for (page, row), s in zip(dest, slots):
            kp[page, row] = k_new[s]
            vp[page, row] = v_new[s]
        plen[r] = P + len(slots)
    return kp, vp, plen, status
