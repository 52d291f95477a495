"""Tiny random candidate pools for exhaustive tests.

Parents are drawn uniformly among earlier local nodes (or the root), so every
tree is topologically ordered.  Log-probabilities come from a small set of
exactly representable values so that path scores tie often.
"""
import numpy as np

TIE_LOGQ = np.array([0.0, -0.5, -1.0, -0.25, -np.inf], dtype=np.float32)


def micro_pool(rng: np.random.Generator, R: int, max_nodes: int, logq_set=TIE_LOGQ,
               p_neg_inf: float = 0.1, vocab: int = 5):
    sizes = rng.integers(0, max_nodes + 1, size=R)
    offs = np.zeros(R + 1, np.int32)
    offs[1:] = np.cumsum(sizes)
    N = int(offs[-1])
    parent = np.empty(N, np.int32)
    token = np.empty(N, np.int32)
    logq = np.empty(N, np.float32)
    finite = logq_set[np.isfinite(logq_set)]
    for r in range(R):
        for n in range(int(sizes[r])):
            g = offs[r] + n
            parent[g] = int(rng.integers(-1, n))            # -1 .. n-1
            token[g] = int(rng.integers(0, vocab))
            if rng.random() < p_neg_inf:
                logq[g] = -np.inf
            else:
                logq[g] = finite[rng.integers(0, len(finite))]
    return dict(cand_offsets=offs, parent=parent, token=token, logq=logq,
                root_token=rng.integers(0, vocab, size=R).astype(np.int32),
                prefix_len=rng.integers(0, 6, size=R).astype(np.int32))
