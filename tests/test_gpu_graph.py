"""Decode and prefill calls captured in HIP graphs, and two handles driven
from two streams at once.

The library's per-call state (router partials, token masks, the plan, the
hand-off counters) lives in the handle and is rebuilt or reset by the calls
themselves, with no memset and no allocation, so a call can be captured once
and replayed.  Each case captures one call on a LLaMA-3-8B-shaped handle and
replays it several times; between replays an eager call of another shape on
the same handle leaves different contents in that state, and unrelated eager
work runs.  Every replay must give the eager call's bits (the decode and
prefill paths are deterministic).
"""
import numpy as np
import pytest

import paper_2605_28283_amd as pp
from paper_2605_28283_amd.workloads import make_layer_device, make_tokens
from gpu_helpers import to_dev

pytestmark = pytest.mark.gpu

D, DFF, E = 4096, 14336, 112

# (mode, T, tau): single-token decode (selection inside the gate/up kernel),
# the sparse headline batch, dense batches (the neuron-tile and grouped gate/up
# kernels, the dense down kernel and its chunk-sum launch), and prefill with
# ragged and full token chunks
CASES = [("decode", 1, 0.5), ("decode", 32, 0.7), ("decode", 64, 0.9), ("decode", 16, 1.0),
         ("decode", 64, 1.0), ("prefill", 700, 0.8), ("prefill", 2048, 0.7)]


@pytest.fixture(scope="module")
def handle():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    pp.load()
    W = make_layer_device(D, DFF, E, 0x6A11)
    h = pp.prunepath_create(D, DFF, E, 2048, W["W_r"], W["W_gate"], W["W_up"], W["W_down"])
    del W
    torch.cuda.synchronize()
    yield h
    pp.prunepath_destroy(h)


def _outputs(torch, T):
    return (torch.empty((T, D), dtype=torch.float32, device="cuda"),
            torch.empty((T, E), dtype=torch.int32, device="cuda"),
            torch.empty((T,), dtype=torch.int32, device="cuda"))


def _call(mode, h, x, T, tau, outs, stream=None):
    fn = pp.prunepath_ffn_decode if mode == "decode" else pp.prunepath_ffn_prefill
    y, idx, cnt = outs
    fn(h, x, T, tau, None, y, idx, cnt, stream=stream)


@pytest.mark.parametrize("mode,T,tau", CASES)
def test_graph_replays_match_eager(handle, mode, T, tau):
    import torch
    print("graph %s T=%d tau=%g" % (mode, T, tau), flush=True)
    x = to_dev(make_tokens(T, D, 300 + T)[0])
    eager = _outputs(torch, T)
    _call(mode, handle, x, T, tau, eager)
    torch.cuda.synchronize()
    ref = [a.cpu().numpy() for a in eager]
    # another shape on the same handle, run eagerly between replays
    om, oT, otau = ("prefill", 300, 0.9) if mode == "decode" else ("decode", 48, 0.6)
    ox = to_dev(make_tokens(oT, D, 77)[0])
    oouts = _outputs(torch, oT)
    g_outs = _outputs(torch, T)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        _call(mode, handle, x, T, tau, g_outs, stream=torch.cuda.current_stream())
    for r in range(3):
        for a in g_outs:
            a.fill_(-3)
        _call(om, handle, ox, oT, otau, oouts)
        junk = torch.randn(1 << 20, device="cuda").sum().item()
        assert np.isfinite(junk)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for name, a, b in zip(("y", "idx", "count"), g_outs, ref):
            assert a.cpu().numpy().tobytes() == b.tobytes(), (mode, T, tau, r, name)
    # the eager call after the replays still gives the same bits
    _call(mode, handle, x, T, tau, eager)
    torch.cuda.synchronize()
    for a, b in zip(eager, ref):
        assert a.cpu().numpy().tobytes() == b.tobytes()


def test_two_handles_on_two_streams(handle):
    """Each handle owns its partials, masks, plan and counters: two handles
    driven from two streams at once (calls interleaved, no synchronisation
    between them) give each handle's sequential results."""
    import torch
    W = make_layer_device(D, DFF, E, 0x6A12)
    h2 = pp.prunepath_create(D, DFF, E, 2048, W["W_r"], W["W_gate"], W["W_up"], W["W_down"])
    del W
    try:
        work = [(handle, "decode", 32, 0.7), (h2, "prefill", 700, 0.8),
                (handle, "decode", 64, 1.0), (h2, "decode", 1, 0.5)]
        xs = [to_dev(make_tokens(T, D, 500 + i)[0]) for i, (_, _, T, _) in enumerate(work)]
        ref = []
        for (h, mode, T, tau), x in zip(work, xs):
            o = _outputs(torch, T)
            _call(mode, h, x, T, tau, o)
            torch.cuda.synchronize()
            ref.append([a.cpu().numpy() for a in o])
        s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
        outs = [_outputs(torch, T) for (_, _, T, _) in work]
        torch.cuda.synchronize()
        for rep in range(3):
            for o in outs:
                for a in o:
                    a.fill_(-5)
            torch.cuda.synchronize()
            # handle's calls in order on s1, h2's on s2, issued alternately
            for (h, mode, T, tau), x, o in zip(work, xs, outs):
                _call(mode, h, x, T, tau, o, stream=s1 if h is handle else s2)
            torch.cuda.synchronize()
            for i, (o, r) in enumerate(zip(outs, ref)):
                for a, b in zip(o, r):
                    assert a.cpu().numpy().tobytes() == b.tobytes(), (rep, i)
    finally:
        pp.prunepath_destroy(h2)
