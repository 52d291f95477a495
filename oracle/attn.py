"""Oracle tree-masked grouped-query verification attention, in float64.

The target model verifies the flattened union of all selected candidates in
one parallel forward pass (Section 3.1, "Super-Tree View").  Inside that
forward each verify slot s of request r, for query head h, attends to

* the request's KV-cache prefix (positions 0 .. P_r-1), and
* the new keys of the request's own slots j whose bit is set in tree_mask[s]
  (s itself and its in-tree ancestors, the root included),

through key/value head h // G with G = Hq / Hkv (consecutive query heads share
a key/value head).  Logits are z_j = sm_scale * <q, k_j>; the output is the
softmax-weighted sum of the visible values and LSE = m + ln(sum exp(z - m)).

Everything is done in float64 on the exactly widened bfloat16 inputs.  A row
that sees no key at all gets output 0 and LSE = -inf.
"""
import numpy as np

from . import status as st


def _bf16_to_f64(bits):
    b = np.asarray(bits, np.uint16).astype(np.uint32) << 16
    return b.view(np.float32).astype(np.float64)


def tree_verify_attn(q, k_new, v_new, k_cache, v_cache, kv_offsets, q_offsets, tree_mask,
                     hq, hkv, sm_scale, rows=None):
    """Return (out float64[Nq, Hq, D], lse float64[Nq, Hq], status).

    q: bf16 bits [cap, Hq, D]; k_new, v_new: [cap, Hkv, D]; k_cache, v_cache:
    [T, Hkv, D]; kv_offsets int64 [R+1]; q_offsets int32 [R+1]; tree_mask
    uint32 [cap, W].  ``rows`` optionally restricts the work to a set of slot
    indices (other rows are left as NaN).
    """
    if hq % hkv != 0:
        raise ValueError("Hq must be a multiple of Hkv")
    G = hq // hkv
    scale = float(np.float32(sm_scale))
    qo = np.asarray(q_offsets, np.int64)
    ko = np.asarray(kv_offsets, np.int64)
    cap = q.shape[0]
    D = q.shape[2]
    R = len(qo) - 1
    status = 0
    nq = int(qo[-1])
    out = np.full((max(nq, 0), hq, D), np.nan)
    lse = np.full((max(nq, 0), hq), np.nan)
    want = None if rows is None else set(int(x) for x in rows)
    for r in range(R):
        q0, q1 = int(qo[r]), int(qo[r + 1])
        k0, k1 = int(ko[r]), int(ko[r + 1])
        if q1 < q0 or q0 < 0 or q1 > cap or k0 < 0 or k1 < k0 or k1 > k_cache.shape[0]:
            status |= st.BAD_OFFSETS
            continue
        n = q1 - q0
        if n == 0:
            continue
        slots = [s for s in range(q0, q1) if want is None or s in want]
        if not slots:
            continue
        for kvh in range(hkv):
            Kp = _bf16_to_f64(k_cache[k0:k1, kvh, :])           # [P, D]
            Vp = _bf16_to_f64(v_cache[k0:k1, kvh, :])
            Kt = _bf16_to_f64(k_new[q0:q1, kvh, :])             # [n, D]
            Vt = _bf16_to_f64(v_new[q0:q1, kvh, :])
            for s in slots:
                # local slots visible to s through the tree mask
                vis = [j for j in range(n)
                       if (int(tree_mask[s, j >> 5]) >> (j & 31)) & 1]
                for h in range(kvh * G, (kvh + 1) * G):
                    qv = _bf16_to_f64(q[s, h, :])
                    z = np.concatenate([scale * (Kp @ qv), scale * (Kt[vis] @ qv)])
                    vals = np.concatenate([Vp, Vt[vis]], axis=0)
                    if z.size == 0:
                        out[s, h] = 0.0
                        lse[s, h] = -np.inf
                        continue
                    m = z.max()
                    w = np.exp(z - m)
                    l = w.sum()
                    out[s, h] = (w @ vals) / l
                    lse[s, h] = m + np.log(l)
    return out, lse, status
