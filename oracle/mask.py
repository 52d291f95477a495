"""Oracle flatten & pack: verify slots, position ids and ancestor bitmasks.

The paper packs the ragged super-tree into a dense, kernel-compatible layout
before the single verification forward (Fig. 3, stage 3 "Flatten & Pack")
but gives no layout.  The layout used here:

* Request r owns the consecutive verify slots [q_offsets[r], q_offsets[r+1]).
  Its local slot 0 is the root (the last verified token, which is always
  re-run); local slots 1.. are its selected candidates in ascending global
  candidate index, so every parent precedes its children.
* slot_parent is request-local (-1 for the root); a candidate whose parent is
  the root points at local slot 0.
* position = P_r + depth, with the root at depth 0 (it sits right after the
  P_r-token KV prefix).
* tree_mask is one row of W uint32 words per slot, least significant bit
  first: bit j of row s (word j >> 5, bit j & 31) is set iff local slot j is
  s itself or one of its ancestors.

If more than B candidates are selected, only the first B in ascending global
index are packed (status OVER_CAPACITY).  A selected node whose parent is not
selected is attached to its nearest selected ancestor (status NOT_CLOSED).
Parent indices outside [-1, local index) met on those walks are read as -1
(status BAD_PARENT).  A malformed candidate CSR (not starting at 0, not ending
at the candidate count, or decreasing) packs the roots only (status
BAD_OFFSETS); that is the library boundary's convention.
"""
import numpy as np

from . import status as st
from .gate import clamped_parents, csr_ok


def build_tree_mask(cand_offsets, parent, token, selected, root_token, prefix_len,
                    budget, mask_words):
    offs = np.asarray(cand_offsets, np.int64)
    R = len(offs) - 1
    budget = int(budget)
    if mask_words * 32 < budget + 1:
        raise ValueError("mask_words too small for budget + 1 slots")
    status = 0
    par_raw = np.asarray(parent, np.int32)
    selected = np.asarray(selected)
    if not csr_ok(offs, len(selected)):
        # malformed candidate CSR: every request keeps its root slot only
        status |= st.BAD_OFFSETS
        selected = np.zeros(len(selected), np.uint8)
        offs = np.zeros(R + 1, np.int64)
        par_raw = np.full(len(selected), -1, np.int32)
    par = clamped_parents(offs, par_raw)
    sel_idx = np.nonzero(selected != 0)[0]
    if len(sel_idx) > budget:
        status |= st.OVER_CAPACITY
        sel_idx = sel_idx[:budget]
    included = np.zeros(int(offs[-1]), bool)
    included[sel_idx] = True

    cap = R + budget
    q_offsets = np.zeros(R + 1, np.int32)
    slot_cand = np.full(cap, -1, np.int32)
    slot_parent = np.full(cap, -1, np.int32)
    slot_token = np.full(cap, -1, np.int32)
    position = np.full(cap, -1, np.int32)
    mask = np.zeros((cap, mask_words), np.uint32)
    for r in range(R):
        lo, hi = int(offs[r]), int(offs[r + 1])
        nodes = [g for g in range(lo, hi) if included[g]]
        base = int(q_offsets[r])
        q_offsets[r + 1] = base + 1 + len(nodes)
        local = {g: 1 + i for i, g in enumerate(nodes)}
        depth = [0] * (1 + len(nodes))
        rows = [[0]]                       # ancestor-or-self sets, by local slot
        slot_cand[base] = -1
        slot_parent[base] = -1
        slot_token[base] = root_token[r]
        position[base] = prefix_len[r]
        for g in nodes:
            j = local[g]
            p = int(par[g])                # request-local candidate index or -1
            if p != par_raw[g]:
                status |= st.BAD_PARENT
            while p >= 0 and (lo + p) not in local:
                status |= st.NOT_CLOSED
                if par[lo + p] != par_raw[lo + p]:
                    status |= st.BAD_PARENT
                p = int(par[lo + p])
            pj = 0 if p < 0 else local[lo + p]
            depth[j] = depth[pj] + 1
            if depth[j] > st.MAX_DEPTH:
                status |= st.TOO_DEEP
            rows.append(rows[pj] + [j])
            slot_cand[base + j] = g
            slot_parent[base + j] = pj
            slot_token[base + j] = token[g]
            position[base + j] = prefix_len[r] + depth[j]
        for j, anc in enumerate(rows):
            for a in anc:
                mask[base + j, a >> 5] |= np.uint32(1 << (a & 31))
    return dict(q_offsets=q_offsets, slot_cand=slot_cand, slot_parent=slot_parent,
                slot_token=slot_token, position_ids=position, tree_mask=mask,
                num_slots=int(q_offsets[-1]), status=status)
