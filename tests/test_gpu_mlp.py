"""GPU parity of the non-gated GELU MLP variant (GPT-2 layers: per-neuron
input bias, output bias once per token) against the fp64 oracle, through the
C ABI, on the same bar as the SwiGLU path: selections bit-exact outside the
tie band, max|y - y_ref| <= 1e-2 RMS(y_ref)."""
import numpy as np
import pytest

import paper_2605_28283_amd as pp
from paper_2605_28283_amd.workloads import (WORKLOADS, make_mlp_layer, make_tokens,
                                            workload_layer, workload_tokens)
from gpu_helpers import DevLayer, parity

pytestmark = pytest.mark.gpu

SIG, STRICT, TOPK, LTE = pp.PP_AGG_SIGMOID, pp.PP_SELECT_STRICT, pp.PP_SELECT_TOPK, pp.PP_SELECT_LTE


@pytest.fixture(scope="module", autouse=True)
def gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    pp.load()
    torch.cuda.init()


@pytest.mark.parametrize("flags", [0, SIG, STRICT, STRICT | SIG])
@pytest.mark.parametrize("mode", ["decode", "prefill"])
def test_mlp_small(oracle_mod, flags, mode):
    """d 512, E 16, biases, ragged batches, the tau sweep with its edges."""
    L = make_mlp_layer(512, 16 * 128, 16, 51)
    with DevLayer(L, 130, flags=flags) as dl:
        for T in (1, 5, 37, 64, 130):
            x, _ = make_tokens(T, 512, 52 + T)
            print("mlp small flags=%d mode=%s T=%d" % (flags, mode, T), flush=True)
            for tau in (0.0, 0.5, 0.9, 1.0):
                parity(oracle_mod, dl, mode, x, tau)


@pytest.mark.parametrize("mode", ["decode", "prefill"])
def test_mlp_permuted_without_biases(oracle_mod, mode):
    """A neuron permutation (the input bias must follow it) and a layer
    created without biases (NULL b_fc, b_proj)."""
    L = make_mlp_layer(1024, 24 * 128, 24, 61, perm=True)
    x, _ = make_tokens(40, 1024, 62)
    with DevLayer(L, 64) as dl:
        for tau in (0.3, 0.8, 1.0):
            parity(oracle_mod, dl, mode, x, tau)
    with DevLayer(L, 64, biases=False) as dl:
        for tau in (0.3, 1.0):
            parity(oracle_mod, dl, mode, x, tau)


@pytest.mark.parametrize("mode", ["decode", "prefill"])
def test_mlp_comparison_rules(oracle_mod, mode):
    """Top-k and the LTE threshold on the MLP kernels; with delta = 1 no
    expert is kept and every row of y is exactly b_proj."""
    L = make_mlp_layer(512, 16 * 128, 16, 71)
    x, _ = make_tokens(33, 512, 72)
    with DevLayer(L, 64, flags=TOPK) as dl:
        for k in (1, 3, 16):
            parity(oracle_mod, dl, mode, x, float(k))
    with DevLayer(L, 64, flags=LTE | SIG) as dl:
        for delta in (0.5, 0.95):
            parity(oracle_mod, dl, mode, x, delta)
        res = parity(oracle_mod, dl, mode, x, 1.0)
        assert (res["cnt"] == 0).all()
        np.testing.assert_array_equal(res["y"], np.tile(L.b_proj, (33, 1)))


@pytest.mark.parametrize("T", [24, 32])
def test_mlp_neuron_tile_units(oracle_mod, T):
    """The non-gated layer on the neuron-tile gate/up units (sparse batch,
    64..96 kept experts of 96 on a 256-CU MI355X): top-6 with expert 0 forced
    into every selection (a group of T > 16 tokens, two token tiles), input
    bias per neuron, output bias once per token; against the oracle."""
    L = make_mlp_layer(1024, 96 * 128, 96, 82)
    L.bias = np.zeros(96, np.float32)
    L.bias[0] = 40.0
    x, _ = make_tokens(T, 1024, 82 + T)
    with DevLayer(L, 64, flags=TOPK | SIG) as dl:
        res = parity(oracle_mod, dl, "decode", x, 6.0)
        assert (res["idx"][:, 0] == 0).all()
        kept = len(set(res["idx"][:, :6].ravel().tolist()))
        print("mlp neuron tiles T=%d: %d kept experts" % (T, kept), flush=True)
        assert 64 <= kept <= 96


@pytest.fixture(scope="module")
def gpt2m():
    w = WORKLOADS["gpt2m_decode"]
    return workload_layer(w), w


def test_mlp_gpt2_medium_decode_sweep(oracle_mod, gpt2m):
    """The GPT-2 Medium MLP shape (d 1024, d_ff 4096, E 32): T x tau sweep
    of the decode workload, every token's selection and y."""
    L, w = gpt2m
    with DevLayer(L, 64) as dl:
        for T in w.T:
            x, _ = workload_tokens(w, T)
            for tau in w.taus:
                print("gpt2m decode T=%d tau=%g" % (T, tau), flush=True)
                parity(oracle_mod, dl, "decode", x, tau)


def test_mlp_gpt2_medium_prefill_matches_decode(oracle_mod, gpt2m):
    """512-token prefill on the GPT-2 Medium shape against the oracle, and
    against the decode path on the same tokens (fp32 summation order only)."""
    L, w = gpt2m
    x, _ = workload_tokens(w, 512, 5)
    with DevLayer(L, 512) as dl:
        a = parity(oracle_mod, dl, "prefill", x, 0.7)
        b = dl.run("decode", x, 0.7)
        np.testing.assert_array_equal(a["idx"], b[0])
        scale = float(np.sqrt(np.mean(b[2].astype(np.float64) ** 2)))
        assert np.abs(a["y"] - b[2]).max() <= 1e-4 * scale


def test_mlp_decode_deterministic(gpt2m):
    L, w = gpt2m
    x, _ = workload_tokens(w, 32, 9)
    with DevLayer(L, 64) as dl:
        a = dl.run("decode", x, 0.9)
        b = dl.run("decode", x, 0.9)
    np.testing.assert_array_equal(a[2], b[2])
