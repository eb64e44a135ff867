"""GPU parity: the HIP path (through the C ABI) against the fp64 oracle.

Selections must match bit for bit except tokens whose cumulative mass (or
logit order at the cut) lies within 1e-5 (counted, checked for validity);
y must satisfy max|y - y_ref| <= 1e-2 * RMS(y_ref), y_ref evaluated by the
oracle on the GPU's own selection.
"""
import numpy as np
import pytest

import paper_2605_28283_amd as pp
from paper_2605_28283_amd.workloads import (WORKLOADS, make_layer, make_tokens, workload_layer,
                                            workload_tokens)
from gpu_helpers import DevLayer, check_output, check_selection, full_size_cap, parity, to_dev

pytestmark = pytest.mark.gpu

NUC, STRICT, SUM, SIG = pp.PP_SELECT_NUCLEUS, pp.PP_SELECT_STRICT, pp.PP_AGG_SUM, pp.PP_AGG_SIGMOID
TOPK, LTE = pp.PP_SELECT_TOPK, pp.PP_SELECT_LTE


@pytest.fixture(scope="module", autouse=True)
def gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    pp.load()
    torch.cuda.init()


@pytest.fixture(scope="module")
def tiny():
    w = WORKLOADS["tiny"]
    return workload_layer(w, 0), w


@pytest.mark.parametrize("flags", [NUC | SUM, NUC | SIG, STRICT | SUM, STRICT | SIG])
@pytest.mark.parametrize("mode", ["decode", "prefill"])
def test_tiny_workload(oracle_mod, tiny, flags, mode):
    L, w = tiny
    x, _ = workload_tokens(w, 4, 0)
    with DevLayer(L, 64, flags) as dl:
        for tau in (0.9, 0.0, 0.3, 0.5, 0.7, 1.0, 1.05):
            parity(oracle_mod, dl, mode, x, tau)


@pytest.mark.parametrize("T", [1, 5, 17, 37, 63, 64, 65, 130])
@pytest.mark.parametrize("mode", ["decode", "prefill"])
def test_ragged_batches(oracle_mod, tiny, T, mode):
    L, _ = tiny
    x, _ = make_tokens(T, L.d, 100 + T)
    with DevLayer(L, 256) as dl:
        for tau in (0.5, 0.9, 1.0):
            parity(oracle_mod, dl, mode, x, tau)


def test_route_entry_point(oracle_mod):
    L = make_layer(512, 2048, 16, 7, skewed=True)
    x, it = make_tokens(23, 512, 8, temperature=True)
    for flags in (NUC | SUM, STRICT | SIG):
        with DevLayer(L, 32, flags) as dl:
            idx, cnt, gw = dl.run("route", x, 0.8, it)
            r, _, _ = check_selection(oracle_mod, L, x, 0.8, flags, idx, cnt, it, label="route")
            for t in range(x.shape[0]):
                k = cnt[t]
                if flags & SIG:
                    exp = 1.0 / (1.0 + np.exp(-r["g"][t, idx[t, :k]]))
                    np.testing.assert_allclose(gw[t, :k], exp, rtol=1e-5, atol=1e-6)
                else:
                    assert (gw[t, :k] == 1.0).all()
                assert (gw[t, k:] == 0.0).all()


@pytest.mark.parametrize("mode", ["decode", "prefill"])
def test_permuted_skewed_medium(oracle_mod, mode):
    """Neuron permutation (Eq. permuted_weights), router bias and temperature,
    several expert tiles (E=24) and a width spanning many K-steps."""
    L = make_layer(1024, 24 * 128, 24, 9, skewed=True, perm=True)
    x, it = make_tokens(50, 1024, 10, temperature=True)
    for flags in (NUC | SUM, STRICT | SIG):
        with DevLayer(L, 64, flags) as dl:
            for tau in (0.5, 0.9, 1.0):
                parity(oracle_mod, dl, mode, x, tau, it)


def test_single_and_max_experts(oracle_mod):
    for E, d, T in ((1, 128, 9), (256, 64, 12), (200, 128, 70)):
        L = make_layer(d, 128 * E, E, 11 + E)
        x, _ = make_tokens(T, d, 12 + E)
        with DevLayer(L, 128) as dl:
            for mode in ("decode", "prefill"):
                for tau in (0.3, 0.9, 1.0):
                    res = parity(oracle_mod, dl, mode, x, tau)
                    if E == 1:
                        assert (res["cnt"] == 1).all()


def test_max_width(oracle_mod):
    """The widest supported d (8192): 16 router K-slices of partial logits and
    256 gate/up K-steps per expert, decode (one token; 70 tokens = a 64-token
    slice plus a ragged 6) and prefill, sparse and dense (tau 1)."""
    d = 8192
    L = make_layer(d, 8 * 128, 8, 31)
    with DevLayer(L, 128) as dl:
        for T in (1, 70):
            x, _ = make_tokens(T, d, 32 + T)
            for mode in ("decode", "prefill"):
                for tau in (0.5, 1.0):
                    parity(oracle_mod, dl, mode, x, tau, label="d=8192 %s" % mode)


@pytest.mark.parametrize("flags,params", [
    (TOPK | SUM, (1, 2, 5, 16, 40)),
    (TOPK | SIG, (3,)),
    (LTE | SUM, (0.0, 0.3, 0.6, 0.9, 0.999, 1.0)),
    (LTE | SIG, (0.5,)),
])
@pytest.mark.parametrize("mode", ["decode", "prefill", "route"])
def test_comparison_rules(oracle_mod, flags, params, mode):
    """Forced top-k and the LTE sigmoid threshold on the same kernels: the
    selections and outputs against the oracle; LTE may keep no expert."""
    L = make_layer(512, 16 * 128, 16, 41)
    x, _ = make_tokens(70, 512, 42)
    with DevLayer(L, 80, flags=flags) as dl:
        for p in params:
            if mode == "route":
                idx, cnt, gw = dl.run("route", x, p)
                r, _, _ = check_selection(oracle_mod, L, x, p, flags, idx, cnt, label="route rules")
                continue
            res = parity(oracle_mod, dl, mode, x, p)
            if flags & LTE and p >= 1.0:
                assert (res["cnt"] == 0).all() and (res["y"] == 0).all()


def test_comparison_rules_llama8b_decode(oracle_mod, llama8b):
    L, w, _ = llama8b
    x, _ = workload_tokens(w, 32, 0)
    for flags, p in ((TOPK, 4), (LTE, 0.95), (STRICT, 0.7)):
        with DevLayer(L, 64, flags=flags) as dl:
            parity(oracle_mod, dl, "decode", x, p, label="llama8b rules")


def test_decode_down_modes_ragged_rows(oracle_mod):
    """d = 576 is not a multiple of 128 or 256: the decode down projection's
    last row block has 64 rows.  tau = 0.3 gives sparse groups (row-tile
    path), tau = 1 keeps every expert (the dense kernel: 128-row units at
    T = 24, 256-row units at T = 64, several expert chunks, summed by their
    own launch), and top-24 of 40 at T = 64 gives ~38 tokens per group
    without keeping every expert (the shared-h dense-group mode, its chunks
    summed by the last to arrive)."""
    L = make_layer(576, 40 * 128, 40, 31)
    for T in (24, 64):
        x, _ = make_tokens(T, 576, 32 + T)
        with DevLayer(L, 64) as dl:
            for tau in (0.3, 1.0):
                a = parity(oracle_mod, dl, "decode", x, tau)
                b = dl.run("decode", x, tau)
                np.testing.assert_array_equal(a["y"], b[2])  # deterministic
        if T == 64:
            with DevLayer(L, 64, flags=TOPK) as dl:
                a = parity(oracle_mod, dl, "decode", x, 24.0)
                assert (a["cnt"] == 24).all()
                b = dl.run("decode", x, 24.0)
                np.testing.assert_array_equal(a["y"], b[2])


@pytest.mark.parametrize("flags", [TOPK, TOPK | SIG])
@pytest.mark.parametrize("T", [24, 32])
def test_decode_neuron_tile_units(oracle_mod, T, flags):
    """Decode batches whose plan takes the neuron-tile gate/up units on a
    256-CU MI355X (sparse groups, between one and one and a half 16-neuron
    tiles per workgroup: 64..96 kept experts): top-6 of 96 experts with
    expert 0 forced into every token's selection by its router bias, so one
    group spans two token tiles (more than 16 tokens) and the others are
    small (70 and 82 kept experts); with the sum and the sigmoid-weighted
    aggregation; against the oracle, deterministic."""
    L = make_layer(1024, 96 * 128, 96, 51)
    L.bias = np.zeros(96, np.float32)
    L.bias[0] = 40.0
    x, _ = make_tokens(T, 1024, 52 + T)
    with DevLayer(L, 64, flags=flags) as dl:
        a = parity(oracle_mod, dl, "decode", x, 6.0)
        assert (a["idx"][:, 0] == 0).all()
        kept = len(set(a["idx"][:, :6].ravel().tolist()))
        print("neuron tiles T=%d: %d kept experts" % (T, kept), flush=True)
        assert 64 <= kept <= 96
        b = dl.run("decode", x, 6.0)
        np.testing.assert_array_equal(a["y"], b[2])


def test_tau_edges_and_counts(oracle_mod, tiny):
    L, _ = tiny
    x, _ = make_tokens(20, L.d, 13)
    with DevLayer(L, 32) as dl:
        _, c0, _ = dl.run("decode", x, 0.0)
        assert (c0 == 1).all()
        _, c1, _ = dl.run("decode", x, 1.0)
        assert (c1 == L.E).all()
        _, c2, _ = dl.run("decode", x, 1.05)
        assert (c2 == L.E).all()
        prev = None
        for tau in np.linspace(0, 1, 21):
            _, c, _ = dl.run("route", x, float(tau))
            if prev is not None:
                assert (c >= prev).all()
            prev = c
    with DevLayer(L, 32, STRICT) as dl:
        _, c, _ = dl.run("decode", x, 1.05)
        assert (c == L.E).all()
        _, c, _ = dl.run("decode", x, 0.0)
        assert (c == 1).all()


def test_invalid_calls_leave_outputs_untouched(tiny):
    import torch
    L, _ = tiny
    x, _ = make_tokens(4, L.d, 14)
    with DevLayer(L, 8) as dl:
        xd = to_dev(x)
        y = torch.full((4, L.d), 3.0, device="cuda")
        idx = torch.full((4, L.E), 5, dtype=torch.int32, device="cuda")
        cnt = torch.full((4,), 5, dtype=torch.int32, device="cuda")
        for T, tau in ((0, 0.5), (9, 0.5), (4, float("nan")), (4, -0.1)):
            for fn in (pp.prunepath_ffn_decode, pp.prunepath_ffn_prefill):
                with pytest.raises(pp.PrunePathError) as ei:
                    fn(dl.h, xd, T, tau, None, y, idx, cnt)
                assert ei.value.status == pp.PP_EINVAL
        with pytest.raises(pp.PrunePathError):
            pp.prunepath_ffn_decode(dl.h, xd, 4, 0.5, None, y, idx, None)
        torch.cuda.synchronize()
        assert (y == 3.0).all() and (idx == 5).all() and (cnt == 5).all()
    bad_perm = torch.zeros(L.d_ff, dtype=torch.int32, device="cuda")
    W = [to_dev(a) for a in (L.W_r, L.W_gate, L.W_up, L.W_down)]
    with pytest.raises(pp.PrunePathError) as ei:
        pp.prunepath_create(L.d, L.d_ff, L.E, 8, *W, perm=bad_perm)
    assert ei.value.status == pp.PP_EINVAL


def test_routing_is_batch_invariant(oracle_mod):
    """A token's selection, and the bits of its gate weights sigmoid(g), do not
    depend on the batch it is routed in (batches above 64 tokens use the
    large-batch logits kernel, smaller ones the per-tile kernel)."""
    L = make_layer(1024, 24 * 128, 24, 17)
    x, _ = make_tokens(200, 1024, 18)
    with DevLayer(L, 256, flags=SIG) as dl:
        full = dl.run("route", x, 0.8)
        for t in (0, 13, 69, 199):
            one = dl.run("route", x[t:t + 1], 0.8)
            np.testing.assert_array_equal(one[0][0], full[0][t])
            assert one[1][0] == full[1][t]
            np.testing.assert_array_equal(one[2][0].view(np.uint32), full[2][t].view(np.uint32))
        for a, b in ((5, 40), (60, 130), (130, 200)):
            part = dl.run("route", x[a:b], 0.8)
            np.testing.assert_array_equal(part[0], full[0][a:b])
            np.testing.assert_array_equal(part[2].view(np.uint32), full[2][a:b].view(np.uint32))


@pytest.mark.parametrize("flags,tau", [(NUC | SIG, 0.8), (STRICT | SUM, 0.8), (TOPK | SIG, 3.0),
                                       (LTE | SUM, 0.9)])
def test_single_token_decode_selects_as_router(oracle_mod, flags, tau):
    """A one-token decode call selects its experts inside the gate/up kernel
    (every workgroup from the partial logits); the selection must equal the
    router's for the same token routed in a batch, and y must pass the oracle
    check."""
    L = make_layer(1024, 24 * 128, 24, 19)
    x, _ = make_tokens(40, 1024, 20)
    with DevLayer(L, 64, flags=flags) as dl:
        full = dl.run("route", x, tau)
        for t in (0, 7, 39):
            idx, cnt, _ = dl.run("decode", x[t:t + 1], tau)
            np.testing.assert_array_equal(idx[0], full[0][t])
            assert cnt[0] == full[1][t]
            parity(oracle_mod, dl, "decode", x[t:t + 1], tau, label="single-token decode")


def test_decode_deterministic_and_matches_prefill(tiny):
    L, _ = tiny
    x, _ = make_tokens(48, L.d, 15)
    with DevLayer(L, 64, STRICT | SIG) as dl:
        a = dl.run("decode", x, 0.8)
        b = dl.run("decode", x, 0.8)
        c = dl.run("prefill", x, 0.8)
    for u, v in zip(a, b):
        np.testing.assert_array_equal(u, v)
    np.testing.assert_array_equal(a[0], c[0])
    np.testing.assert_array_equal(a[1], c[1])
    rms = np.sqrt(np.mean(a[2].astype(np.float64) ** 2))
    assert np.abs(a[2] - c[2]).max() <= 1e-4 * rms


# ------------------------------------------------------------------ full-size workloads

@pytest.fixture(scope="module")
def llama8b():
    w = WORKLOADS["llama8b_decode"]
    L = workload_layer(w, 0)
    dl = DevLayer(L, 2048)
    yield L, w, dl
    dl.close()


@pytest.mark.parametrize("T", [1, 8, 32, 64])
def test_llama8b_decode_sweep(oracle_mod, llama8b, T):
    """Full LLaMA-3-8B FFN shape, the decode launch configuration the benchmark
    times: every token's selection and every row of y against the oracle."""
    L, w, dl = llama8b
    x, _ = workload_tokens(w, 64, 0)
    x = x[:T]
    for tau in w.taus:
        parity(oracle_mod, dl, "decode", x, tau, label="llama8b decode",
               max_exempt=full_size_cap(T))


def test_llama8b_prefill(oracle_mod, llama8b):
    """2048-token prefill at the benchmark's taus: every selection and every
    row of y (four full 512-token chunks of the down projection) against the
    oracle; the decode path agrees with prefill on the same tokens."""
    L, _, dl = llama8b
    w = WORKLOADS["llama8b_prefill"]
    x, _ = workload_tokens(w, 2048, 0)
    for tau in w.taus:
        res = parity(oracle_mod, dl, "prefill", x, tau, label="llama8b prefill",
                     max_exempt=full_size_cap(2048))
        # decode path on the same tokens agrees with prefill everywhere
        idx, cnt, y = dl.run("decode", x, tau)
        np.testing.assert_array_equal(idx, res["idx"])
        rms = np.sqrt(np.mean(res["y"].astype(np.float64) ** 2))
        assert np.abs(y - res["y"]).max() <= 1e-3 * rms


def test_llama8b_prefill_many_pairs(oracle_mod, llama8b):
    """Over 100k (token, expert) pairs in one call, with very uneven tokens:
    even tokens route nearly flat (inverse temperature 0.01: most experts kept
    at tau 0.95), odd tokens sharply (inverse temperature 20: one or two
    kept), so the experts' runs in each 512-token chunk are long and every
    expert's down block meets tokens of both kinds.  y: the whole first
    512-token chunk and both sides of every chunk edge."""
    L, w, dl = llama8b
    T = 2048
    x, _ = make_tokens(T, w.d, 91)
    it = np.where(np.arange(T) % 2 == 0, 0.01, 20.0).astype(np.float32)
    rows = np.concatenate([np.arange(512), [1023, 1024, 1535, 1536, 2046, 2047]])
    res = parity(oracle_mod, dl, "prefill", x, 0.95, it, rows=rows, label="prefill many pairs")
    assert int(res["cnt"].sum()) > 65536
    assert res["cnt"][1::2].max() <= 8


def test_llama8b_prefill_ragged_chunks(oracle_mod, llama8b):
    """700 tokens: one full 512-token chunk of the down projection and a ragged
    one (the 32-row units); every row of y against the oracle."""
    L, w, dl = llama8b
    x, _ = make_tokens(700, w.d, 93, row_lognormal_sigma=0.5)
    parity(oracle_mod, dl, "prefill", x, 0.8, label="prefill 700 tokens",
           max_exempt=full_size_cap(700))


def test_qwen_skewed(oracle_mod):
    """The wide skewed-routing layer (d 3584, E 148, Gumbel router bias,
    per-token temperature), T = 64: every selection and every row of y."""
    w = WORKLOADS["qwen7b_skewed"]
    L = workload_layer(w, 0)
    x, it = workload_tokens(w, 64, 0)
    with DevLayer(L, 64) as dl:
        for tau in w.taus:
            res = parity(oracle_mod, dl, "decode", x, tau, it, label="qwen7b skewed",
                         max_exempt=full_size_cap(64))
            assert res["cnt"].min() >= 1


def test_prefill_deterministic(oracle_mod, llama8b):
    """Prefill sums each token's expert contributions in a fixed order (no
    float atomics): reruns give the same bits."""
    L, w, dl = llama8b
    x, _ = make_tokens(300, w.d, 77, row_lognormal_sigma=0.5)
    a = dl.run("prefill", x, 0.8)
    b = dl.run("prefill", x, 0.8)
    np.testing.assert_array_equal(a[2], b[2])
    np.testing.assert_array_equal(a[0], b[0])
