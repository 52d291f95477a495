"""The timed attention entry points: events recorded around the main kernel of
that one call, on that call's stream, and outputs equal to the untimed call."""
import numpy as np
import pytest

import synth
from tests import gpu_common as gc

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _need_gpu():
    gc.require_gpu()


@pytest.mark.parametrize("page_size", [None, 64])
def test_two_streams_time_independently(page_size):
    import torch
    from paper_2604_09603_amd.step import VerifyStep
    b = synth.make_batch("l8b", 2)
    ref = gc.oracle_front(b)
    print(f"[timing] l8b seed 2, page size {page_size}", flush=True)
    steps = [VerifyStep(b, page_size=page_size) for _ in range(2)]
    for st in steps:
        st.set_target(ref["target"])
    steps[0].run()
    base = steps[0].fetch()
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    events = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
              for _ in range(2)]
    # torch reads the time of an event it has recorded itself: record each once
    for (a, c), s in zip(events, streams):
        a.record(s)
        c.record(s)
    torch.cuda.synchronize()
    for st, s, ev in zip(steps, streams, events):
        with torch.cuda.stream(s):
            st.gate()
            st.mask()
            st.attn(events=ev)
            st.accept()
    torch.cuda.synchronize()
    for st, (a, c) in zip(steps, events):
        ms = a.elapsed_time(c)
        assert 0.0 < ms < 100.0, ms
        res = st.fetch()
        nq = res["num_slots"]
        assert nq == base["num_slots"]
        assert np.array_equal(res["out"][:nq].view(np.uint32), base["out"][:nq].view(np.uint32))
        assert np.array_equal(res["lse"][:nq].view(np.uint32), base["lse"][:nq].view(np.uint32))
        assert np.array_equal(res["accept_len"], base["accept_len"])
    # a second timed call on one stream re-records its own pair only
    (a0, c0), (a1, c1) = events
    t_other = a1.elapsed_time(c1)
    with torch.cuda.stream(streams[0]):
        steps[0].attn(events=(a0, c0))
    torch.cuda.synchronize()
    assert a1.elapsed_time(c1) == t_other
    assert a0.elapsed_time(c0) > 0.0


def test_stream_read_probe_runs():
    """The read-ceiling probe in both modes over a small token-major cache."""
    import torch
    import paper_2604_09603_amd as pkg
    d = torch.device("cuda:0")
    rows, heads = 4096 + 17, 4
    k = torch.randint(-2**15, 2**15 - 1, (rows, heads, 128), dtype=torch.int16, device=d)
    v = torch.randint(-2**15, 2**15 - 1, (rows, heads, 128), dtype=torch.int16, device=d)
    sink = torch.zeros(1, dtype=torch.int32, device=d)
    for mode in (0, 1):
        pkg.echo_probe_stream_read(k, v, rows, heads, mode, sink)
    pkg.echo_probe_stream_read(k, v, rows - 17, heads, 2, sink)
    torch.cuda.synchronize()
