"""Oracle gate: path scores and the global budgeted top-B selection.

Path score (eq. 5, Section 3.2 "Path Scoring"): for a draft node j at depth d
with parent pa(j), S_j = S_pa(j) + log q(x_j | h_pa(j)), with S = 0 at the
root.  The recursion runs from the root towards the leaves, one IEEE binary32
addition per level, exactly in that order.

Selection (eq. 4, Section 3.1 "Super-Tree View"): the whole batch shares one
verification cap, sum_i K_i <= K_max = B draft nodes.  Which nodes to spend it
on follows the marginal-utility exchange of Theorem 2 with the objective of
Proposition 1 (Appendix, "Batch-Level Objective"): the node-level marginal
gain of verifying node j is its path confidence exp(S_j) (eq. 6 uses the same
quantity as the confidence of a depth), and because log q <= 0 makes S
non-increasing along every root-to-leaf path, repeatedly moving a unit of
budget to a larger exp(S) ends at the B candidates with the largest S.  That
set is closed under taking parents.  Ties in S go to the smaller global
candidate index; -inf (a pruned or impossible node) is never selected.
"""
import numpy as np

from . import status as st


def csr_ok(cand_offsets, N):
    """A candidate CSR is usable iff it starts at 0, ends at N and never decreases.

    This is the library boundary's convention, not the paper's: a malformed CSR
    is a data error (BAD_OFFSETS), no candidate is scored and none is selected.
    """
    offs = np.asarray(cand_offsets, np.int64)
    return int(offs[0]) == 0 and int(offs[-1]) == int(N) and bool(np.all(np.diff(offs) >= 0))


def path_scores(cand_offsets, parent, logq):
    """S per candidate (float32), depth per candidate (root's children: 1), status.

    ``cand_offsets`` is the request-major CSR (R+1 entries); ``parent`` holds
    request-local indices (-1 = child of the root).  Clamps: NaN log q -> -inf,
    log q > 0 -> 0, parent outside [-1, local index) -> -1, depth > MAX_DEPTH ->
    S = -inf.  A malformed CSR (see ``csr_ok``) gives S = -inf everywhere.
    """
    offs = np.asarray(cand_offsets, np.int64)
    parent = np.asarray(parent, np.int32)
    logq = np.asarray(logq, np.float32)
    N = len(logq)
    S = np.full(N, -np.inf, np.float32)
    depth = np.zeros(N, np.int32)
    status = 0
    if not csr_ok(offs, N):
        return S, depth, st.BAD_OFFSETS
    zero = np.float32(0.0)
    for r in range(len(offs) - 1):
        lo, hi = int(offs[r]), int(offs[r + 1])
        for n in range(hi - lo):
            g = lo + n
            p = int(parent[g])
            if p < -1 or p >= n:
                status |= st.BAD_PARENT
                p = -1
            lq = logq[g]
            if np.isnan(lq):
                status |= st.NAN_LOGQ
                lq = np.float32(-np.inf)
            elif lq > 0:
                status |= st.POS_LOGQ
                lq = zero
            if p < 0:
                base, d = zero, 1
            else:
                base, d = S[lo + p], int(depth[lo + p]) + 1
            s = np.float32(base + lq)            # one binary32 add, root -> leaf
            if d > st.MAX_DEPTH:
                status |= st.TOO_DEEP
                s = np.float32(-np.inf)
            S[g] = s
            depth[g] = d
    return S, depth, status


def select_top_b(S, budget):
    """Boolean mask of the min(B, #finite) largest S (ties -> smaller index)."""
    S = np.asarray(S, np.float32)
    finite = np.nonzero(np.isfinite(S))[0]
    # primary key: S descending (-0 and +0 compare equal); secondary: index ascending
    order = finite[np.lexsort((finite, -S[finite].astype(np.float64)))]
    take = order[:min(int(budget), len(finite))]
    sel = np.zeros(len(S), np.uint8)
    sel[take] = 1
    return sel


def clamped_parents(cand_offsets, parent):
    offs = np.asarray(cand_offsets, np.int64)
    out = np.asarray(parent, np.int32).copy()
    for r in range(len(offs) - 1):
        lo, hi = int(offs[r]), int(offs[r + 1])
        for n in range(hi - lo):
            if out[lo + n] < -1 or out[lo + n] >= n:
                out[lo + n] = -1
    return out


def gate(cand_offsets, parent, logq, budget):
    """Full gate: returns dict(path_score, selected, num_selected, status)."""
    S, depth, status = path_scores(cand_offsets, parent, logq)
    sel = select_top_b(S, budget)
    if not csr_ok(cand_offsets, len(S)):
        return dict(path_score=S, depth=depth, selected=sel, num_selected=0, status=status)
    # ancestor closure: every selected node's parent is selected
    offs = np.asarray(cand_offsets, np.int64)
    par = clamped_parents(cand_offsets, parent)
    for r in range(len(offs) - 1):
        lo, hi = int(offs[r]), int(offs[r + 1])
        for g in range(lo, hi):
            if sel[g] and par[g] >= 0 and not sel[lo + par[g]]:
                status |= st.NOT_CLOSED
    return dict(path_score=S, depth=depth, selected=sel,
                num_selected=int(sel.sum()), status=status)
