"""Exhaustive and dense reference computations used to pin the oracle.

Everything here is written independently of ``oracle/``: path scores are
exact rational sums over explicitly enumerated root paths, the gate is an
exhaustive search over ancestor-closed subsets, masks come from a dense
transitive closure, attention is one dense masked softmax over every key of
the batch, and acceptance enumerates every root-to-slot path.
"""
import itertools
import math
from fractions import Fraction

import numpy as np


def root_path(offs, parent, g):
    """Global indices on the path root -> g (excluding the root), using raw parents."""
    r = int(np.searchsorted(offs, g, side="right") - 1)
    lo = int(offs[r])
    path = [g]
    while int(parent[path[-1]]) >= 0:
        path.append(lo + int(parent[path[-1]]))
    return path[::-1]


def exact_path_score(offs, parent, logq, g):
    """Exact sum of log q along the root path (None for -inf)."""
    tot = Fraction(0)
    for x in root_path(offs, parent, g):
        v = float(logq[x])
        if v == -math.inf:
            return None
        tot += Fraction(v)
    return tot


def closed(offs, parent, subset):
    s = set(subset)
    for g in subset:
        r = int(np.searchsorted(offs, g, side="right") - 1)
        p = int(parent[g])
        if p >= 0 and int(offs[r]) + p not in s:
            return False
    return True


def brute_gate(offs, parent, logq, budget):
    """Ancestor-closed subset of size min(B, #finite) maximising sum exp(S);
    among maximisers the lexicographically smallest sorted index tuple."""
    N = int(offs[-1])
    S = {g: exact_path_score(offs, parent, logq, g) for g in range(N)}
    finite = [g for g in range(N) if S[g] is not None]
    m = min(budget, len(finite))
    best, best_val = None, None
    for comb in itertools.combinations(finite, m):
        if not closed(offs, parent, comb):
            continue
        val = math.fsum(math.exp(float(S[g])) for g in comb)
        if best is None or val > best_val + 1e-12 * abs(best_val) or (
                abs(val - best_val) <= 1e-12 * abs(best_val) and comb < best):
            best, best_val = comb, val
    return set(best if best is not None else ()), S


def transitive_closure(parent_local):
    """Dense ancestor-or-self matrix from local parent pointers (Warshall)."""
    n = len(parent_local)
    A = np.eye(n, dtype=bool)
    for s, p in enumerate(parent_local):
        if p >= 0:
            A[s, p] = True
    for k in range(n):
        A |= A[:, [k]] & A[[k], :]
    return A


def unpack_mask(row_words, n):
    return np.array([(int(row_words[j >> 5]) >> (j & 31)) & 1 for j in range(n)], bool)


def dense_attention(q, k_new, v_new, k_cache, v_cache, kv_offsets, q_offsets, vis_tree, hq, hkv,
                    sm_scale):
    """One dense masked softmax per (slot, head) over every key of the whole batch.

    vis_tree[s] is a set of global slot indices whose new keys slot s sees.
    """
    f = lambda b: (np.asarray(b, np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    G = hq // hkv
    R = len(q_offsets) - 1
    nq = int(q_offsets[-1])
    T = int(kv_offsets[-1])
    Kall = np.concatenate([f(k_cache[:T]), f(k_new[:nq])], axis=0)   # [T + nq, Hkv, D]
    Vall = np.concatenate([f(v_cache[:T]), f(v_new[:nq])], axis=0)
    out = np.zeros((nq, hq, q.shape[2]))
    lse = np.zeros((nq, hq))
    for r in range(R):
        for s in range(int(q_offsets[r]), int(q_offsets[r + 1])):
            allowed = np.zeros(T + nq, bool)
            allowed[int(kv_offsets[r]):int(kv_offsets[r + 1])] = True
            for j in vis_tree[s]:
                allowed[T + j] = True
            for h in range(hq):
                kvh = h // G
                z = float(np.float32(sm_scale)) * (Kall[:, kvh, :] @ f(q[s, h]))
                z = np.where(allowed, z, -np.inf)
                if not allowed.any():
                    out[s, h] = 0.0
                    lse[s, h] = -np.inf
                    continue
                m = z.max()
                p = np.exp(z - m)
                out[s, h] = (p @ Vall[:, kvh, :]) / p.sum()
                lse[s, h] = m + math.log(p.sum())
    return out, lse


def brute_accept(n, slot_parent_local, tokens, targets, max_depth):
    """Enumerate every root->slot path of one request; return (len, end, path)."""
    best = (0, 0, [])
    for s in range(n):
        path = [s]
        ok = True
        while path[-1] != 0:
            p = slot_parent_local[path[-1]]
            if p < 0 or p >= path[-1]:
                ok = False
                break
            path.append(p)
        if not ok:
            continue
        path = path[::-1]
        d = len(path) - 1
        if d > max_depth:
            continue
        if all(tokens[path[i + 1]] == targets[path[i]] for i in range(d)):
            if d > best[0] or (d == best[0] and s < best[1]):
                best = (d, s, path[1:])
    return best
