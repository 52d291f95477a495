"""Oracle elastic budget scheduler: Alg. 1 (Section 3.3, "Unified Elastic Budget
Scheduling") as a selection policy over an already-drafted candidate pool.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The scheduler walks the draft depths in order and serves the requests of the
batch from one shared budget K_max (eq. 4):

* Phase 1, global depth extension (priority 1).  At depth d = 1, 2, ... every
  still-active request, in request order and while budget remains, is tested
  at the checkpoint depths (eq. 7, with the layer confidence of eq. 6 taken
  over the depth-d candidates it could append).  A request that passes appends
  its W_topk best depth-d candidates and pays for them; one that fails leaves
  the active set for the truncated set.  The phase ends when the budget is
  spent or no request is active.
* Phase 2, opportunistic width expansion (priority 2).  With budget left, each
  truncated request widens the last depth it kept, up to W_max nodes there.

Readings (the listing is garbled in places; each choice is the plain one):

* Candidates of request i at depth d are its depth-d nodes whose parent it
  already holds (the root for d = 1) and whose path score is finite; "best"
  is (S descending, global index ascending), the order of the top-B gate.
* c_{i,d} > tau_d is tested as max S > ln tau_d in binary32 (eq. 6 without the
  exp); a depth with no candidate has c = 0 and fails a checkpoint.  Depths
  that are not checkpoints always pass.
* An append takes min(W_topk, budget left, #candidates) nodes and is charged
  what it takes, so the total never exceeds K_max.  A request that passes but
  has no candidate has exhausted its drafted tree: it leaves the active set
  without being truncated.  Depth stops at MAX_DEPTH.
* Phase 2 serves the truncated requests in request order.  A request
  truncated at depth t widens depth t - 1 (nothing if t = 1: the root cannot
  be widened) by w = min(budget left, W_max - its width there, #remaining
  candidates there) and is charged w.
"""
import numpy as np

from . import status as st
from .gate import clamped_parents, csr_ok, path_scores


def _best(cands, S, k):
    """The k best candidates by (S descending, index ascending)."""
    order = sorted(cands, key=lambda g: (-float(S[g]), g))
    return order[:max(0, k)]


def elastic_schedule(cand_offsets, parent, logq, budget, sig_depth, log_tau, w_topk, w_max):
    """Returns dict(path_score, selected, num_selected, status, trunc_depth, width).

    ``trunc_depth[i]`` is the depth at which request i failed a checkpoint
    during phase 1 (MAX_DEPTH + 1 if it never did); ``width[i, d]`` the number
    of its nodes selected at depth d.
    """
    S, depth, status = path_scores(cand_offsets, parent, logq)
    offs = np.asarray(cand_offsets, np.int64)
    R = len(offs) - 1
    N = len(S)
    sel = np.zeros(N, np.uint8)
    width = np.zeros((R, st.MAX_DEPTH + 1), np.int32)
    trunc_depth = np.full(R, st.MAX_DEPTH + 1, np.int32)
    if not csr_ok(offs, N):
        return dict(path_score=S, selected=sel, num_selected=0, status=status,
                    trunc_depth=trunc_depth, width=width)
    par = clamped_parents(offs, parent)
    lt_at = {}
    for d, lt in zip(sig_depth, log_tau):   # a depth listed twice must pass both
        d = int(d)
        lt_at[d] = max(lt_at.get(d, -np.inf), float(np.float32(lt)))

    def candidates(i, d):
        lo, hi = int(offs[i]), int(offs[i + 1])
        return [g for g in range(lo, hi)
                if depth[g] == d and np.isfinite(S[g]) and not sel[g]
                and (par[g] < 0 or sel[lo + par[g]])]

    left = int(budget)
    active = list(range(R))
    truncated = []
    d = 0
    # Phase 1: global depth extension
    while left > 0 and active and d < st.MAX_DEPTH:
        d += 1
        for i in list(active):
            if left <= 0:
                break
            cands = candidates(i, d)
            if d in lt_at:
                c = max((S[g] for g in cands), default=np.float32(-np.inf))
                passed = bool(np.float32(c) > np.float32(lt_at[d]))
            else:
                passed = True
            if not passed:
                active.remove(i)
                truncated.append(i)
                trunc_depth[i] = d
                continue
            if not cands:
                active.remove(i)        # drafted tree exhausted
                continue
            take = _best(cands, S, min(int(w_topk), left))
            for g in take:
                sel[g] = 1
            width[i, d] += len(take)
            left -= len(take)
    # Phase 2: opportunistic width expansion of the truncated requests
    for i in sorted(truncated):
        if left <= 0:
            break
        lvl = int(trunc_depth[i]) - 1
        if lvl < 1:
            continue
        room = int(w_max) - int(width[i, lvl])
        take = _best(candidates(i, lvl), S, min(room, left))
        for g in take:
            sel[g] = 1
        width[i, lvl] += len(take)
        left -= len(take)
    # closure holds by construction; checked like the top-B gate
    for r in range(R):
        lo, hi = int(offs[r]), int(offs[r + 1])
        for g in range(lo, hi):
            if sel[g] and par[g] >= 0 and not sel[lo + par[g]]:
                status |= st.NOT_CLOSED
    return dict(path_score=S, selected=sel, num_selected=int(sel.sum()), status=status,
                trunc_depth=trunc_depth, width=width)
