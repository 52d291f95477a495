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


# ---------------------------------------------------------------------------
# Sparse gating at checkpoint depths (Section 3.2, eq. 6 and eq. 7; Alg. 1).
#
# Layer confidence (eq. 6): c_{i,d} = exp(max over request i's depth-d nodes
# of S).  Gating signal (eq. 7): g_{i,d} = [c_{i,d} > tau_d], evaluated only
# at the calibrated checkpoint depths d in D_sig.  The comparison is taken in
# the log domain, max S > ln tau_d, with ln tau_d supplied by the caller as a
# float32 (exp is monotone, so this is the same test without an exp).
#
# Reading of the truncation (Alg. 1, phase 1): the scheduler walks the depths
# in order and a request whose checkpoint test fails at depth d leaves the
# active set before its depth-d tokens are appended, so none of its nodes at
# depth >= d is verified.  The freed budget returns to the shared pool, which
# the global top-B of eq. 4 then spends on the remaining nodes (other
# requests' depth, or this request's width above d).  Depths that are not
# checkpoints always pass.
# ---------------------------------------------------------------------------

def layer_max_scores(cand_offsets, S, depth):
    """max S per (request, depth): array [R, MAX_DEPTH + 1] of float32, -inf
    where a request has no node (or only -inf nodes) at that depth.  Column 0
    (the root) is unused.  This is eq. 6 before the exp."""
    offs = np.asarray(cand_offsets, np.int64)
    R = len(offs) - 1
    out = np.full((R, st.MAX_DEPTH + 1), -np.inf, np.float32)
    if not csr_ok(offs, len(S)):
        return out
    for r in range(R):
        for g in range(int(offs[r]), int(offs[r + 1])):
            d = int(depth[g])
            if 1 <= d <= st.MAX_DEPTH and S[g] > out[r, d]:
                out[r, d] = S[g]
    return out


def truncation_depths(layer_max, sig_depth, log_tau):
    """First failing checkpoint per request (eq. 7), MAX_DEPTH + 1 if none fails.

    Checkpoint k sits at depth sig_depth[k] with threshold ln tau = log_tau[k];
    request i fails it iff NOT (layer_max[i, d] > log_tau[k]) in float32.
    """
    R = layer_max.shape[0]
    t = np.full(R, st.MAX_DEPTH + 1, np.int32)
    for i in range(R):
        for d, lt in zip(sig_depth, log_tau):
            d = int(d)
            passed = bool(np.float32(layer_max[i, d]) > np.float32(lt))
            if not passed and d < t[i]:
                t[i] = d
    return t


def gate_sparse(cand_offsets, parent, logq, budget, sig_depth, log_tau):
    """Sparse-gated selection: the checkpoint truncation of eq. 7, then the
    global top-B of eq. 4 over the nodes that survive it.

    Returns the dict of ``gate`` plus ``trunc_depth`` [R] (first failing
    checkpoint, MAX_DEPTH + 1 if none) and ``layer_max`` [R, MAX_DEPTH + 1].
    ``path_score`` is the untruncated eq. 5 score.
    """
    S, depth, status = path_scores(cand_offsets, parent, logq)
    offs = np.asarray(cand_offsets, np.int64)
    R = len(offs) - 1
    lm = layer_max_scores(offs, S, depth)
    t = truncation_depths(lm, sig_depth, log_tau)
    S_gate = S.copy()
    if csr_ok(offs, len(S)):
        for r in range(R):
            for g in range(int(offs[r]), int(offs[r + 1])):
                if depth[g] >= t[r]:
                    S_gate[g] = -np.inf
    sel = select_top_b(S_gate, budget)
    if not csr_ok(offs, len(S)):
        return dict(path_score=S, depth=depth, selected=sel, num_selected=0, status=status,
                    trunc_depth=t, layer_max=lm)
    par = clamped_parents(offs, parent)
    for r in range(R):
        lo, hi = int(offs[r]), int(offs[r + 1])
        for g in range(lo, hi):
            if sel[g] and par[g] >= 0 and not sel[lo + par[g]]:
                status |= st.NOT_CLOSED
    return dict(path_score=S, depth=depth, selected=sel, num_selected=int(sel.sum()),
                status=status, trunc_depth=t, layer_max=lm)
