"""Device-resident buffers for one verification step and the four calls in order.

``VerifyStep`` owns every input, output and workspace of a batch on one GPU
(torch allocations, used only as device memory) and enqueues echo_gate ->
echo_build_tree_mask -> echo_tree_verify_attn -> echo_accept on the current
stream, or the same four stages as one echo_verify_step call (``run_fused``).  The target argmax per verify slot is an input of the last stage; the
caller supplies it (``set_target``) because it comes from the target model.
"""
import numpy as np
import torch

from . import (HEAD_DIM, MAX_DEPTH, echo_accept, echo_accept_logits, echo_build_tree_mask,
               echo_commit_kv, echo_gate, echo_gate_elastic, echo_gate_sparse,
               echo_tree_verify_attn, echo_tree_verify_attn_paged,
               echo_tree_verify_attn_paged_timed, echo_tree_verify_attn_timed, echo_verify_step,
               gate_elastic_workspace_size, gate_workspace_size, tree_verify_attn_workspace_size)


def _aligned_workspace(nbytes, device):
    raw = torch.empty(max(int(nbytes), 1) + 256, dtype=torch.uint8, device=device)
    off = (-raw.data_ptr()) % 256
    return raw[off:off + max(int(nbytes), 1)]


def _dev(a, device, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(a))
    if dtype is not None:
        t = t.to(dtype)
    return t.to(device)


class VerifyStep:
    """``checkpoints``: optional sequence of (depth, ln tau) pairs; when given the
    gate stage is echo_gate_sparse (checkpoint truncation, then top-B).
    ``elastic``: optional (w_topk, w_max); when given the gate stage is
    echo_gate_elastic (Alg. 1) with the checkpoints (none if not given).
    ``page_size``: optional; the KV prefixes are then scattered over shuffled
    pages of that many rows (with room for the commits of one step) and the
    attention stage is echo_tree_verify_attn_paged.
    ``serve``: with ``page_size``, acceptance reads the target argmax from
    logits (``set_logits``) and each step ends with echo_commit_kv; the cached
    lengths are restored afterwards so that every step repeats the same work."""

    def __init__(self, batch, device="cuda:0", max_depth=MAX_DEPTH, checkpoints=None,
                 elastic=None, page_size=None, serve=False, page_seed=0):
        cfg = batch["cfg"]
        self.checkpoints = None if checkpoints is None else [(int(d), float(t))
                                                             for d, t in checkpoints]
        self.elastic = None if elastic is None else (int(elastic[0]), int(elastic[1]))
        self.cfg = cfg
        self.device = device
        self.R = cfg.R
        self.N = int(batch["cand_offsets"][-1])
        self.B = cfg.budget
        self.cap = cfg.R + cfg.budget
        self.W = (cfg.budget + 1 + 31) // 32
        self.hq, self.hkv, self.D = cfg.hq, cfg.hkv, cfg.head_dim
        self.max_depth = max_depth
        d = device
        i16 = lambda a: _dev(np.asarray(a, np.uint16).view(np.int16), d)
        # inputs
        self.cand_offsets = _dev(batch["cand_offsets"].astype(np.int32), d)
        self.parent = _dev(batch["parent"].astype(np.int32), d)
        self.token = _dev(batch["token"].astype(np.int32), d)
        self.logq = _dev(batch["logq"].astype(np.float32), d)
        self.root_token = _dev(batch["root_token"].astype(np.int32), d)
        self.prefix_len = _dev(batch["prefix_len"].astype(np.int32), d)
        self.kv_offsets = _dev(batch["kv_offsets"].astype(np.int64), d)
        self.kv_rows = int(batch["kv_offsets"][-1])
        self.q = i16(batch["q"])
        self.k_new = i16(batch["k_new"])
        self.v_new = i16(batch["v_new"])
        self.k_cache = i16(batch["k_cache"])
        self.v_cache = i16(batch["v_cache"])
        self.sm_scale = float(batch["sm_scale"])
        self.page_size = None if page_size is None else int(page_size)
        self.serve = bool(serve)
        if self.serve and self.page_size is None:
            raise ValueError("the serving step needs a paged cache (page_size)")
        if self.page_size is not None:
            self._make_pages(batch, page_seed)
        # outputs
        z32 = lambda *s: torch.zeros(s, dtype=torch.int32, device=d)
        self.path_score = torch.zeros(max(self.N, 1), dtype=torch.float32, device=d)
        self.selected = torch.zeros(max(self.N, 1), dtype=torch.uint8, device=d)
        self.num_selected = z32(1)
        self.trunc_depth = z32(self.R)
        self.q_offsets = z32(self.R + 1)
        self.slot_cand = z32(self.cap)
        self.slot_parent = z32(self.cap)
        self.slot_token = z32(self.cap)
        self.position_ids = z32(self.cap)
        self.tree_mask = z32(self.cap, self.W)
        self.out = torch.zeros((self.cap, self.hq, self.D), dtype=torch.float32, device=d)
        self.lse = torch.zeros((self.cap, self.hq), dtype=torch.float32, device=d)
        self.target_token = z32(self.cap)
        self.accept_len = z32(self.R)
        self.accept_slots = z32(self.R, max_depth)
        self.bonus_token = z32(self.R)
        self.status = z32(1)
        ws_size = (gate_elastic_workspace_size if self.elastic is not None else gate_workspace_size)
        self.gate_ws = _aligned_workspace(ws_size(self.R, self.N, self.B), d)
        self.attn_ws = _aligned_workspace(
            tree_verify_attn_workspace_size(self.R, self.cap, self.hq, self.hkv, self.D), d)

    def _make_pages(self, batch, seed):
        """Scatter every prefix over shuffled pages; each request also gets the
        pages its commit of one step (at most 1 + max_depth rows) can reach."""
        S = self.page_size
        P = np.asarray(batch["prefix_len"], np.int64)
        kvo = np.asarray(batch["kv_offsets"], np.int64)
        npg = (P + 1 + self.max_depth + S - 1) // S
        total = int(npg.sum())
        perm = np.random.default_rng(seed).permutation(total).astype(np.int64)
        bt = np.full((self.R, int(npg.max())), -1, np.int32)
        dest = np.empty(int(kvo[-1]), np.int64)
        k = 0
        for r in range(self.R):
            ids = perm[k:k + npg[r]]
            k += npg[r]
            bt[r, :npg[r]] = ids
            pos = np.arange(P[r])
            dest[kvo[r]:kvo[r + 1]] = ids[pos // S] * S + pos % S
        d = self.device
        shape = (total, S, self.hkv, self.D)
        self.k_pages = torch.zeros(shape, dtype=torch.int16, device=d)
        self.v_pages = torch.zeros(shape, dtype=torch.int16, device=d)
        idx = torch.from_numpy(dest).to(d)
        self.k_pages.view(total * S, self.hkv, self.D)[idx] = self.k_cache
        self.v_pages.view(total * S, self.hkv, self.D)[idx] = self.v_cache
        self.block_table = _dev(bt, d)
        self.cached_len = self.prefix_len.clone()   # grows with commits
        self.logits = None
        self.target_out = torch.zeros(self.cap, dtype=torch.int32, device=d)

    def set_logits(self, logits):
        """bf16 target logits [cap, V] (torch.bfloat16 or int16 bits) on the device."""
        self.logits = logits.view(torch.int16) if logits.dtype == torch.bfloat16 else logits

    # ---- the four stages -------------------------------------------------
    def gate(self, stream=None):
        if self.elastic is not None:
            ck = self.checkpoints or []
            echo_gate_elastic(self.cand_offsets, self.parent, self.logq, self.R, self.N, self.B,
                              [d for d, _ in ck], [t for _, t in ck], self.elastic[0],
                              self.elastic[1], self.path_score, self.selected, self.num_selected,
                              self.gate_ws, trunc_depth=self.trunc_depth, status=self.status,
                              stream=stream)
        elif self.checkpoints is None:
            echo_gate(self.cand_offsets, self.parent, self.logq, self.R, self.N, self.B,
                      self.path_score, self.selected, self.num_selected, self.gate_ws,
                      status=self.status, stream=stream)
        else:
            echo_gate_sparse(self.cand_offsets, self.parent, self.logq, self.R, self.N, self.B,
                             [d for d, _ in self.checkpoints], [t for _, t in self.checkpoints],
                             self.path_score, self.selected, self.num_selected, self.gate_ws,
                             trunc_depth=self.trunc_depth, status=self.status, stream=stream)

    def mask(self, stream=None):
        echo_build_tree_mask(self.cand_offsets, self.parent, self.token, self.selected,
                             self.root_token, self.prefix_len, self.R, self.N, self.B,
                             self.q_offsets, self.slot_cand, self.slot_parent, self.slot_token,
                             self.position_ids, self.tree_mask, self.W, status=self.status,
                             stream=stream)

    def attn(self, stream=None, events=None):
        """``events``: optional (start, stop) torch.cuda.Event pair recorded around the
        main attention kernel (the timed entry points; measurement only)."""
        if self.page_size is not None:
            args = (self.q, self.k_new, self.v_new, self.k_pages, self.v_pages, self.page_size,
                    self.block_table, self.cached_len, self.q_offsets, self.tree_mask, self.W,
                    self.R, self.cap, self.hq, self.hkv, self.D, self.sm_scale, self.out,
                    self.lse, self.attn_ws)
            if events is None:
                echo_tree_verify_attn_paged(*args, status=self.status, stream=stream)
            else:
                echo_tree_verify_attn_paged_timed(*args, events[0], events[1],
                                                  status=self.status, stream=stream)
            return
        args = (self.q, self.k_new, self.v_new, self.k_cache, self.v_cache, self.kv_offsets,
                self.kv_rows, self.q_offsets, self.tree_mask, self.W, self.R, self.cap, self.hq,
                self.hkv, self.D, self.sm_scale, self.out, self.lse, self.attn_ws)
        if events is None:
            echo_tree_verify_attn(*args, status=self.status, stream=stream)
        else:
            echo_tree_verify_attn_timed(*args, events[0], events[1], status=self.status,
                                        stream=stream)

    def accept(self, stream=None):
        if self.serve:
            echo_accept_logits(self.q_offsets, self.slot_parent, self.slot_token, self.logits,
                               self.R, self.cap, self.max_depth, self.target_out,
                               self.accept_len, self.accept_slots, self.bonus_token,
                               status=self.status, stream=stream)
            return
        echo_accept(self.q_offsets, self.slot_parent, self.slot_token, self.target_token, self.R,
                    self.cap, self.max_depth, self.accept_len, self.accept_slots,
                    self.bonus_token, status=self.status, stream=stream)

    def commit(self, stream=None):
        echo_commit_kv(self.q_offsets, self.accept_len, self.accept_slots, self.max_depth,
                       self.k_new, self.v_new, self.R, self.cap, self.hkv, self.k_pages,
                       self.v_pages, self.page_size, self.block_table, self.cached_len,
                       status=self.status, stream=stream)

    def fused_ok(self):
        """The one-call step covers the top-B gate, a contiguous cache and acceptance
        from target tokens."""
        return (self.elastic is None and self.checkpoints is None and self.page_size is None
                and not self.serve)

    def run_fused(self, stream=None):
        """The step as one echo_verify_step call (same outputs as run())."""
        if not self.fused_ok():
            raise ValueError("echo_verify_step covers the top-B gate on a contiguous cache")
        echo_verify_step(self.cand_offsets, self.parent, self.logq, self.token, self.R, self.N,
                         self.B, self.path_score, self.selected, self.num_selected, self.gate_ws,
                         self.root_token, self.prefix_len, self.q_offsets, self.slot_cand,
                         self.slot_parent, self.slot_token, self.position_ids, self.tree_mask,
                         self.W, self.q, self.k_new, self.v_new, self.k_cache, self.v_cache,
                         self.kv_offsets, self.kv_rows, self.cap, self.hq, self.hkv, self.D,
                         self.sm_scale, self.out, self.lse, self.attn_ws, self.target_token,
                         self.max_depth, self.accept_len, self.accept_slots, self.bonus_token,
                         status=self.status, stream=stream)

    def run(self, stream=None, attn_events=None):
        self.gate(stream)
        self.mask(stream)
        self.attn(stream, attn_events)
        self.accept(stream)
        if self.serve:
            self.commit(stream)
            # the next step repeats this one: forget the committed rows
            with torch.cuda.stream(stream if stream is not None else torch.cuda.current_stream()):
                self.cached_len.copy_(self.prefix_len, non_blocking=True)

    def set_target(self, target_per_slot):
        t = np.zeros(self.cap, np.int32)
        t[:len(target_per_slot)] = target_per_slot
        self.target_token.copy_(torch.from_numpy(t))

    def fetch(self):
        torch.cuda.synchronize()
        g = lambda t: t.cpu().numpy()
        nq = int(self.q_offsets[-1].item())
        return dict(
            path_score=g(self.path_score)[:self.N], selected=g(self.selected)[:self.N],
            num_selected=int(self.num_selected.item()), trunc_depth=g(self.trunc_depth),
            q_offsets=g(self.q_offsets),
            slot_cand=g(self.slot_cand), slot_parent=g(self.slot_parent),
            slot_token=g(self.slot_token), position_ids=g(self.position_ids),
            tree_mask=g(self.tree_mask).view(np.uint32), out=g(self.out), lse=g(self.lse),
            accept_len=g(self.accept_len), accept_slots=g(self.accept_slots),
            bonus_token=g(self.bonus_token), status=int(self.status.item()), num_slots=nq)
