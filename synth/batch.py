"""Seeded synthetic batches shaped like one speculative-decoding verification step.

This module only draws random inputs.  It holds none of the verification
arithmetic (no path scores, no selection, no masks, no attention, no
acceptance): both the CPU oracle and the GPU library consume what it returns.

Recipe (per request r, one numpy PCG64 stream per request, spawned from
``SeedSequence(seed)``):

* Draft tree ("beam" shape, the drafter stand-in).  The root is expanded by
  drawing logits z ~ N(0,1)*sigma over the vocabulary V; its top-k tokens
  (ties -> lower token id) become the depth-1 nodes, with
  logq = log_softmax(z)[token] in float32.  For depth d = 2..D the k nodes of
  depth d-1 that come first in the order (frontier rank of the parent +
  sibling rank, sibling rank, parent rank) are expanded the same way, so depth
  d holds k*k nodes.  Nodes are stored in level order, so a parent always has
  a smaller local index than its children, and N_r = k + (D-1)*k*k.  The
  frontier is ranked by integer ranks only; the confidence arithmetic stays
  in the gate.
* Target model stand-in.  For every expanded node x (the root included) the
  target argmax after x equals the token of x's top-1 child with probability
  p_r and is otherwise uniform over the other V-1 tokens; after a node that
  was not expanded it is uniform over V.  p_r is the preset's constant or is
  drawn per request from its Beta distribution.
* Attention tensors.  Prefix lengths P_r ~ UniformInt[p_lo, p_hi]; q, k_new,
  v_new (slot-indexed, R+B capacity rows) and the token-major KV cache are
  N(0,1) rounded to bfloat16 (round to nearest even), stored as uint16 bit
  patterns.
"""
from __future__ import annotations

import os
import zlib
from concurrent.futures import ThreadPoolExecutor

import numpy as np

from .configs import CONFIGS, Config

_THREADS = max(1, min(16, os.cpu_count() or 1))


def _salt(cfg: Config) -> int:
    return zlib.crc32(cfg.name.encode())


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (nearest even); return the uint16 bit patterns."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    rnd = ((b >> 16) & 1) + np.uint32(0x7FFF)
    return ((b + rnd) >> 16).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def _expand(rng: np.random.Generator, vocab: int, k: int, sigma: float):
    """One drafter expansion: top-k tokens of N(0,1)*sigma logits and their log-softmax."""
    z = rng.standard_normal(vocab, dtype=np.float32)
    if k < vocab:
        part = np.argpartition(z, vocab - k)[vocab - k:]
        thr = z[part].min()
        cand = np.nonzero(z >= thr)[0]          # includes every tie at the boundary
    else:
        cand = np.arange(vocab)
    order = np.lexsort((cand, -z[cand]))        # value desc, token id asc
    top = cand[order][:k]
    m = z.max()
    s = np.exp((z - m) * np.float32(sigma)).sum(dtype=np.float64)
    lse = float(m) * sigma + np.log(s)
    logq = (z[top].astype(np.float64) * sigma - lse).astype(np.float32)
    return top.astype(np.int32), logq


def _draw_target(rng, vocab, top1):
    """Uniform token over the vocabulary without ``top1`` (or over all of it if top1 < 0)."""
    if top1 < 0:
        return int(rng.integers(0, vocab))
    u = int(rng.integers(0, vocab - 1))
    return u if u < top1 else u + 1


def _request_tree(ss: np.random.SeedSequence, cfg: Config):
    rng = np.random.Generator(np.random.PCG64(ss))
    k, D, V = cfg.branch, cfg.depth, cfg.vocab
    if cfg.accept[0] == "const":
        p_acc = float(cfg.accept[1])
    else:
        p_acc = float(rng.beta(cfg.accept[1], cfg.accept[2]))
    parent, token, logq, top1 = [], [], [], []
    root_tok = int(rng.integers(0, V))
    top, lq = _expand(rng, V, k, cfg.sigma)
    root_top1 = int(top[0])
    for c in range(k):
        parent.append(-1); token.append(int(top[c])); logq.append(lq[c]); top1.append(-1)
    # frontier entries: (local node index, frontier rank)
    level = [(i, 0, c) for c, i in enumerate(range(k))]   # (node, parent rank, sibling rank)
    for d in range(2, D + 1):
        level.sort(key=lambda t: (t[1] + t[2], t[2], t[1]))
        frontier = [t[0] for t in level[:k]]
        nxt = []
        for prank, f in enumerate(frontier):
            top, lq = _expand(rng, V, k, cfg.sigma)
            top1[f] = int(top[0])
            for c in range(k):
                nxt.append((len(parent), prank, c))
                parent.append(f); token.append(int(top[c])); logq.append(lq[c]); top1.append(-1)
        level = nxt
    # target argmax after each node (stand-in for the target model's LM head)
    def tgt(t1):
        if t1 >= 0 and rng.random() < p_acc:
            return t1
        return _draw_target(rng, V, t1)
    root_target = tgt(root_top1)
    target = [tgt(t) for t in top1]
    return dict(parent=np.asarray(parent, np.int32), token=np.asarray(token, np.int32),
                logq=np.asarray(logq, np.float32), target=np.asarray(target, np.int32),
                root_token=root_tok, root_target=root_target, p_accept=p_acc)


def _normal_bf16(ss: np.random.SeedSequence, n: int, chunk: int = 1 << 22) -> np.ndarray:
    """n N(0,1) values rounded to bf16, drawn in fixed chunks (thread-count independent)."""
    out = np.empty(n, dtype=np.uint16)
    nch = (n + chunk - 1) // chunk
    seeds = ss.spawn(nch)

    def fill(i):
        lo, hi = i * chunk, min(n, (i + 1) * chunk)
        rng = np.random.Generator(np.random.PCG64(seeds[i]))
        out[lo:hi] = f32_to_bf16_bits(rng.standard_normal(hi - lo, dtype=np.float32))

    with ThreadPoolExecutor(_THREADS) as ex:
        list(ex.map(fill, range(nch)))
    return out


def make_trees(cfg: Config, seed: int):
    """The drafted candidate pool of every request, as a request-major CSR."""
    ss_tree = np.random.SeedSequence([seed, 0, _salt(cfg)]).spawn(cfg.R)
    with ThreadPoolExecutor(_THREADS) as ex:
        reqs = list(ex.map(lambda s: _request_tree(s, cfg), ss_tree))
    sizes = np.array([len(r["parent"]) for r in reqs], np.int64)
    offs = np.zeros(cfg.R + 1, np.int32)
    offs[1:] = np.cumsum(sizes)
    cat = lambda key, dt: np.concatenate([r[key] for r in reqs]).astype(dt)
    return dict(
        cand_offsets=offs,
        parent=cat("parent", np.int32),
        token=cat("token", np.int32),
        logq=cat("logq", np.float32),
        target=cat("target", np.int32),
        root_token=np.array([r["root_token"] for r in reqs], np.int32),
        root_target=np.array([r["root_target"] for r in reqs], np.int32),
        p_accept=np.array([r["p_accept"] for r in reqs], np.float64),
    )


def _scaled(bits: np.ndarray, scale: float) -> np.ndarray:
    return bits if scale == 1.0 else f32_to_bf16_bits(bf16_bits_to_f32(bits) * np.float32(scale))


def make_attention_inputs(cfg: Config, seed: int, q_scale: float = 1.0, v_scale: float = 1.0):
    """Prefix lengths, slot-indexed q/k_new/v_new and the token-major KV cache (bf16 bits).
    q_scale / v_scale multiply the queries / the values (new and cached) after the
    draw, rounded back to bf16."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 1, _salt(cfg)])))
    P = rng.integers(cfg.p_lo, cfg.p_hi + 1, size=cfg.R).astype(np.int32)
    kv_offsets = np.zeros(cfg.R + 1, np.int64)
    kv_offsets[1:] = np.cumsum(P.astype(np.int64))
    cap, D = cfg.capacity, cfg.head_dim
    qkv_ss = np.random.SeedSequence([seed, 2, _salt(cfg)]).spawn(5)
    q = _scaled(_normal_bf16(qkv_ss[0], cap * cfg.hq * D), q_scale)
    k_new = _normal_bf16(qkv_ss[1], cap * cfg.hkv * D)
    v_new = _scaled(_normal_bf16(qkv_ss[2], cap * cfg.hkv * D), v_scale)
    T = int(kv_offsets[-1])
    k_cache = _normal_bf16(qkv_ss[3], T * cfg.hkv * D)
    v_cache = _scaled(_normal_bf16(qkv_ss[4], T * cfg.hkv * D), v_scale)
    return dict(
        prefix_len=P, kv_offsets=kv_offsets,
        q=q.reshape(cap, cfg.hq, D), k_new=k_new.reshape(cap, cfg.hkv, D),
        v_new=v_new.reshape(cap, cfg.hkv, D),
        k_cache=k_cache.reshape(T, cfg.hkv, D), v_cache=v_cache.reshape(T, cfg.hkv, D),
        sm_scale=np.float32(1.0 / np.sqrt(D)),
    )


def make_batch(name_or_cfg, seed: int, attention: bool = True, q_scale: float = 1.0,
               v_scale: float = 1.0):
    cfg = CONFIGS[name_or_cfg] if isinstance(name_or_cfg, str) else name_or_cfg
    b = dict(cfg=cfg, seed=seed)
    b.update(make_trees(cfg, seed))
    if attention:
        b.update(make_attention_inputs(cfg, seed, q_scale, v_scale))
    return b


def target_for_slots(batch, q_offsets: np.ndarray, slot_cand: np.ndarray) -> np.ndarray:
    """Target argmax per verify slot: the stand-in for the target model's output.

    Slot 0 of request r is its root; other slots carry the global candidate index.
    """
    R = len(q_offsets) - 1
    nq = int(q_offsets[-1])
    out = np.empty(nq, np.int32)
    for r in range(R):
        lo, hi = int(q_offsets[r]), int(q_offsets[r + 1])
        if hi > lo:
            out[lo] = batch["root_target"][r]
            if hi > lo + 1:
                out[lo + 1:hi] = batch["target"][slot_cand[lo + 1:hi]]
    return out
