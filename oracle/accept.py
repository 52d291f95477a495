"""Oracle greedy acceptance over each request's verified slot tree.

Speculative decoding accepts the longest drafted prefix the target agrees
with (Section 2, "Standard SD"), and the target always contributes one more
token of its own (the "+1" of eq. 1).  The paper runs greedy decoding
(temperature 0, Section 5.1 and the evaluation details), so a draft token is
accepted exactly when it equals the target argmax computed after its parent.
On a tree:

* the root (local slot 0) is always valid;
* slot s is valid iff its parent is valid, its depth is at most max_depth and
  slot_token[s] == target_token[parent(s)];
* the accepted path ends at the valid slot of largest depth, ties to the
  smallest local slot; accept_len is that depth, accept_slots lists the
  path's global slot indices from depth 1 down to the end slot (-1 padded to
  max_depth entries) and bonus_token = target_token[end slot].

A request without slots gets accept_len 0, bonus -1.  slot_parent outside
[0, s) makes slot s (and its subtree) unacceptable (status BAD_SLOT_PARENT).
"""
import numpy as np

from . import status as st


def accept(q_offsets, slot_parent, slot_token, target_token, max_depth):
    qo = np.asarray(q_offsets, np.int64)
    R = len(qo) - 1
    cap = len(slot_parent)
    status = 0
    acc_len = np.zeros(R, np.int32)
    acc_slots = np.full((R, max_depth), -1, np.int32)
    bonus = np.full(R, -1, np.int32)
    for r in range(R):
        lo, hi = int(qo[r]), int(qo[r + 1])
        if hi < lo or lo < 0 or hi > cap:
            status |= st.BAD_OFFSETS
            continue
        n = hi - lo
        if n == 0:
            continue
        valid = [False] * n
        depth = [0] * n
        par = [-1] * n
        valid[0] = True
        for s in range(1, n):
            p = int(slot_parent[lo + s])
            if p < 0 or p >= s:
                status |= st.BAD_SLOT_PARENT
                continue
            par[s] = p
            depth[s] = depth[p] + 1
            valid[s] = (valid[p] and depth[s] <= max_depth
                        and int(slot_token[lo + s]) == int(target_token[lo + p]))
        end = 0
        for s in range(1, n):
            if valid[s] and depth[s] > depth[end]:
                end = s
        path = []
        s = end
        while s > 0:
            path.append(lo + s)
            s = par[s]
        path.reverse()
        acc_len[r] = depth[end]
        acc_slots[r, :len(path)] = path
        bonus[r] = target_token[lo + end]
    return dict(accept_len=acc_len, accept_slots=acc_slots, bonus_token=bonus, status=status)
