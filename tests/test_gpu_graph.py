"""The whole step captured in a HIP graph (through torch.cuda.CUDAGraph) and
replayed: every replay, with eager work and synchronisations in between, must
reproduce the eager step bit for bit (the library records no memset nodes)."""
import sys

import numpy as np
import pytest

import synth
from tests import gpu_common as gc

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _need_gpu():
    gc.require_gpu()


KEYS = ["path_score", "selected", "num_selected", "q_offsets", "slot_cand", "slot_parent",
        "slot_token", "position_ids", "tree_mask", "accept_len", "accept_slots", "bonus_token",
        "status"]


def _same(a, b, nq):
    for k in KEYS:
        assert np.array_equal(np.asarray(a[k]), np.asarray(b[k])), k
    for k in ("out", "lse"):
        assert np.array_equal(a[k][:nq].view(np.uint32), b[k][:nq].view(np.uint32)), k


@pytest.mark.parametrize("name,mode", [("tiny", "plain"), ("l8b", "plain"), ("l8b", "sparse"),
                                       ("l8b", "elastic"), ("tiny", "serve"), ("l70b", "serve")])
def test_graph_replays_match_eager(name, mode):
    import torch
    from paper_2604_09603_amd.step import VerifyStep
    print(f"[graph] {name} {mode}", flush=True)
    b = synth.make_batch(name, 1)
    ref = gc.oracle_front(b)
    kw = {}
    if mode in ("sparse", "elastic"):
        kw["checkpoints"] = [(1, -3.0), (3, -8.0)]
    if mode == "elastic":
        kw["elastic"] = (2, 8)
    if mode == "serve":
        kw.update(page_size=64, serve=True)
    st = VerifyStep(b, **kw)
    st.set_target(ref["target"])
    if mode == "serve":
        gen = torch.Generator(device="cuda:0")
        gen.manual_seed(7)
        logits = torch.randn((st.cap, b["cfg"].vocab), generator=gen, device="cuda:0")
        st.set_logits(logits.to(torch.bfloat16))
    st.run()
    eager = st.fetch()
    nq = eager["num_slots"]
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        st.run()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        st.run()
    torch.cuda.synchronize()
    for i in range(4):
        # poison the outputs eagerly, do unrelated eager work, then replay
        st.out.fill_(float("nan"))
        st.selected.fill_(9)
        st.accept_len.fill_(-3)
        x = torch.randn(256, 256, device="cuda:0")
        (x @ x).sum().item()
        graph.replay()
        got = st.fetch()
        _same(got, eager, nq)
        if mode == "serve":
            assert torch.equal(st.cached_len, st.prefix_len)
    print(f"[graph] {name} {mode}: 4 replays equal the eager step", flush=True)
