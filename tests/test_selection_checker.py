"""CPU checks of the selection-parity checker used by the GPU tests
(tests/gpu_helpers.check_selection): it must accept exactly what the tie
readings allow and reject everything else.  Logits are planted exactly: the
tokens are one-hot (x = e_0) and column 0 of W_r holds the logits, all
bf16-representable, so g = W_r x is exact in any precision."""
import types

import numpy as np
import pytest

import gpu_helpers
from gpu_helpers import check_selection
from paper_2605_28283_amd.workloads import bf16_bits as f32_to_bf16


@pytest.fixture(autouse=True)
def keep_tie_log_for_gpu_calls():
    """The terminal summary reports the GPU parity calls only."""
    n = len(gpu_helpers.TIE_LOG)
    yield
    del gpu_helpers.TIE_LOG[n:]


def layer(logit_rows):
    """One token per row of logits: returns (layer stub, x bits)."""
    G = np.asarray(logit_rows, np.float32)
    T, E = G.shape
    # token t is e_t; W_r[:, t] holds token t's logits
    W = np.zeros((E, T), np.float32)
    W[:, :] = G.T
    x = np.eye(T, dtype=np.float32)
    L = types.SimpleNamespace(W_r=f32_to_bf16(W), bias=None)
    return L, f32_to_bf16(x)


def sel(idx_rows, E):
    idx = np.full((len(idx_rows), E), -1, np.int32)
    for t, r in enumerate(idx_rows):
        idx[t, :len(r)] = r
    return idx, np.array([len(r) for r in idx_rows], np.int32)


def run(oracle_mod, L, x, tau, rows, flags=0):
    idx, cnt = sel(rows, L.W_r.shape[0])
    return check_selection(oracle_mod, L, x, tau, flags, idx, cnt, label="checker")


def test_exact_selection_passes_and_counts_nothing(oracle_mod):
    L, x = layer([[4.0, 1.0, 0.0, -2.0]])
    r, ex, c = run(oracle_mod, L, x, 0.5, [[0]])
    assert c["exempt"] == 0 and not ex.any()


def test_wrong_set_or_count_fails(oracle_mod):
    L, x = layer([[2.0, 1.5, 0.0, -2.0]])
    # tau = 0.7: the oracle keeps {0, 1}
    run(oracle_mod, L, x, 0.7, [[0, 1]])
    for bad in ([[0]], [[0, 2]], [[0, 1, 2]]):
        with pytest.raises(AssertionError):
            run(oracle_mod, L, x, 0.7, bad)


def test_order_swap_only_between_tied_logits(oracle_mod):
    # experts 1 and 2 tie exactly inside the kept prefix
    L, x = layer([[3.0, 2.0, 2.0, -4.0, -4.0]])
    # tau = 0.95: C_2 = 0.787, C_3 = 0.999, so the oracle keeps [0, 1, 2]
    r, ex, c = run(oracle_mod, L, x, 0.95, [[0, 2, 1]])  # tied pair listed the other way
    assert list(r["idx"][0, :3]) == [0, 1, 2]
    assert c["prefix_order"] == 1 and c["exempt"] == 0
    with pytest.raises(AssertionError):  # an untied pair swapped
        run(oracle_mod, L, x, 0.95, [[1, 0, 2]])


def test_cut_tie_may_keep_either(oracle_mod):
    # experts 1 and 2 tie exactly at the cut of tau = 0.85: C_1 = 0.785,
    # C_2 = 0.892, so k = 2 and the oracle keeps [0, 1]
    L, x = layer([[3.0, 1.0, 1.0, -3.0]])
    r, ex, c = run(oracle_mod, L, x, 0.85, [[0, 2]])
    assert list(r["idx"][0, :2]) == [0, 1]
    assert c["cut_order"] == 1 and c["exempt"] == 1
    r, ex, c = run(oracle_mod, L, x, 0.85, [[0, 1]])
    with pytest.raises(AssertionError):  # an exempt token must still be a valid prefix
        run(oracle_mod, L, x, 0.85, [[0, 3]])


def test_mass_tie_count_range(oracle_mod):
    # two experts of equal logit: C_1 = 0.5 exactly; tau = 0.5 is a mass tie,
    # so k = 1 and k = 2 are both valid, k = 3 is not
    L, x = layer([[1.0, 1.0, -30.0]])
    for rows in ([[0]], [[0, 1]]):
        r, ex, c = run(oracle_mod, L, x, 0.5, rows)
        assert c["mass"] == 1
    with pytest.raises(AssertionError):
        run(oracle_mod, L, x, 0.5, [[0, 1, 2]])


def test_cap_on_exempt_tokens(oracle_mod):
    L, x = layer([[3.0, 1.0, 1.0, -3.0], [3.0, 1.0, 1.0, -3.0], [4.0, 0.0, -1.0, -3.0]])
    idx, cnt = sel([[0, 1], [0, 2], [0]], 4)
    check_selection(oracle_mod, L, x, 0.85, 0, idx, cnt, max_exempt=2)
    with pytest.raises(AssertionError):
        check_selection(oracle_mod, L, x, 0.85, 0, idx, cnt, max_exempt=1)
