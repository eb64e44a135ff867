"""Pins of the CPU oracle against things other than itself.

Each check ties one part of the oracle (Sec. 3.1 routing, Sec. 2.1/2.2 expert
evaluation) to a library routine, a closed form, brute force or the paper's
exact identity (Eq. moefication_decomp: all experts reproduce the dense FFN).
Chosen so that a dropped term, a wrong sign, a swapped operand or an index
slip anywhere in the oracle fails at least one of them.
"""
import itertools
import math
import os

import numpy as np
import pytest
from scipy.special import softmax as sp_softmax

from paper_2605_28283_amd.workloads import bf16_bits, bf16_to_f32, make_layer, make_tokens

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "select_worked_cases.txt")


def f64(bits):
    return bf16_to_f32(bits).astype(np.float64)


def silu(a):
    return a / (1.0 + np.exp(-a))


def dense_ffn(x, Wg, Wu, Wd):
    """Eq. (ffn) with the API's [out, in] layouts, numpy float64, no experts."""
    X, G, U, D = f64(x), f64(Wg), f64(Wu), f64(Wd)
    return (silu(X @ G.T) * (X @ U.T)) @ D.T


def small_layer(d=64, E=6, seed=3, perm=False, skewed=False):
    return make_layer(d, 128 * E, E, seed, perm=perm, skewed=skewed)


# ---------------------------------------------------------------- routing steps

def test_logits_match_numpy_matmul(oracle_mod):
    L = small_layer(d=96, E=12, skewed=True)
    x, it = make_tokens(7, 96, 11, temperature=True)
    r = oracle_mod.route(x, L.W_r, 0.9, bias=L.bias, inv_temp=it)
    ref = (f64(x) @ f64(L.W_r).T + L.bias.astype(np.float64)) * it.astype(np.float64)[:, None]
    np.testing.assert_allclose(r["g"], ref, rtol=1e-12, atol=1e-12)
    # and without the extras the bias / temperature must not leak in
    r0 = oracle_mod.route(x, L.W_r, 0.9)
    np.testing.assert_allclose(r0["g"], f64(x) @ f64(L.W_r).T, rtol=1e-12, atol=1e-12)


def test_softmax_textbook(oracle_mod):
    rng = np.random.default_rng(5)
    for E in (1, 2, 16, 112, 256):
        g = rng.normal(0, 3, E) + 40.0  # offset: must be shift-invariant
        p = oracle_mod.softmax(g)
        np.testing.assert_allclose(p, sp_softmax(g), rtol=1e-13, atol=1e-300)
        assert abs(p.sum() - 1.0) < 1e-14


def test_order_matches_stable_argsort(oracle_mod):
    rng = np.random.default_rng(6)
    for E in (1, 3, 16, 112, 256):
        g = np.round(rng.normal(0, 2, E), 1)  # rounding creates exact ties
        pi = oracle_mod.order(g)
        np.testing.assert_array_equal(pi, np.argsort(-g, kind="stable"))


def nucleus_ref(C, tau):
    E = len(C)
    if tau >= 1.0:
        return E
    for i in range(E):
        if C[i] >= tau:
            return i + 1
    return E


def test_cut_closed_form(oracle_mod):
    rng = np.random.default_rng(7)
    for trial in range(50):
        E = int(rng.integers(1, 40))
        p = np.sort(rng.dirichlet(np.full(E, 0.3)))[::-1]
        for tau in np.concatenate([[0.0, 1.0, 1.05], rng.uniform(0, 1, 8)]):
            k, C = oracle_mod.cut(p, tau, 0)
            np.testing.assert_allclose(C, np.cumsum(p), rtol=1e-14)
            assert 1 <= k <= E
            if tau < 1.0 and k < E:
                assert C[k - 1] >= tau
            if k > 1 and tau < 1.0:
                assert C[k - 2] < tau
            if tau >= 1.0:
                assert k == E
            assert k == nucleus_ref(C, tau)
    # tau = 1 keeps every expert even when the float cumulative sum saturates
    # at 1 before the tail (every softmax probability is positive)
    p = np.array([1.0, 1e-20, 1e-30])
    assert oracle_mod.cut(p, 1.0, 0)[0] == 3
    assert oracle_mod.cut(p, 1.0 - 1e-12, 0)[0] == 1


def test_strict_relation(oracle_mod):
    """The printed rule keeps one expert fewer than the nucleus prefix for
    0 < tau < 1, never fewer than one, and all E only for tau > 1."""
    rng = np.random.default_rng(8)
    for trial in range(50):
        E = int(rng.integers(2, 40))
        p = np.sort(rng.dirichlet(np.full(E, 0.5)))[::-1]
        for tau in rng.uniform(0.01, 0.99, 6):
            kn, C = oracle_mod.cut(p, tau, 0)
            ks, _ = oracle_mod.cut(p, tau, 1)
            if np.min(np.abs(C - tau)) < 1e-12:
                continue
            assert ks == max(1, kn - 1)
        kn1, C = oracle_mod.cut(p, 1.0, 1)
        assert kn1 == int(np.sum(C[:-1] < 1.0))
        assert oracle_mod.cut(p, 1.05, 1)[0] == E
        assert oracle_mod.cut(p, 0.0, 1)[0] == 1


def test_brute_force_small_E(oracle_mod):
    """E <= 8: the nucleus set is a minimum-cardinality subset reaching tau
    and has the largest mass among subsets of that size."""
    rng = np.random.default_rng(9)
    for trial in range(40):
        E = int(rng.integers(2, 9))
        g = rng.normal(0, 2, E)
        p = sp_softmax(g)
        tau = float(rng.uniform(0.05, 0.99))
        pi = oracle_mod.order(g)
        k, C = oracle_mod.cut(p[pi], tau, 0)
        if np.min(np.abs(C - tau)) < 1e-12:
            continue
        best_card, best_mass = None, {}
        for r in range(1, E + 1):
            for sub in itertools.combinations(range(E), r):
                m = p[list(sub)].sum()
                best_mass[r] = max(best_mass.get(r, 0.0), m)
                if m >= tau and best_card is None:
                    best_card = r
        assert k == best_card
        assert abs(p[pi[:k]].sum() - best_mass[k]) < 1e-12


def _golden_cases():
    out = []
    with open(GOLDEN) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            kind, vals, tau, rule, exp = [s.strip() for s in line.split("|")]
            out.append((kind, [float(v) for v in vals.split()], float(tau), rule,
                        [int(v) for v in exp.split()]))
    return out


def test_golden_worked_cases(oracle_mod):
    cases = _golden_cases()
    assert len(cases) >= 20
    for kind, vals, tau, rule, expected in cases:
        flags = oracle_mod.SELECT_STRICT if rule == "strict" else 0
        if kind == "probs":
            p = np.array(vals)
            pi = oracle_mod.order(np.log(p))
            k, _ = oracle_mod.cut(p[pi], tau, flags)
            got = list(pi[:k])
        else:
            E = len(vals)
            x = bf16_bits(np.array([[1.0]], np.float32))
            W_r = bf16_bits(np.array(vals, np.float32).reshape(E, 1))
            r = oracle_mod.route(x, W_r, tau, flags)
            got = list(r["idx"][0, : r["count"][0]])
        assert got == expected, (kind, vals, tau, rule)


def test_route_selection_vs_numpy(oracle_mod):
    L = small_layer(d=128, E=16, seed=4)
    x, _ = make_tokens(40, 128, 12)
    for tau in (0.0, 0.3, 0.5, 0.8, 0.95, 1.0, 1.05):
        r = oracle_mod.route(x, L.W_r, tau)
        g = f64(x) @ f64(L.W_r).T
        for t in range(x.shape[0]):
            order = np.argsort(-g[t], kind="stable")
            C = np.cumsum(sp_softmax(g[t])[order])
            k = nucleus_ref(C, tau)
            assert r["count"][t] == k
            np.testing.assert_array_equal(r["idx"][t, :k], order[:k])
            assert (r["idx"][t, k:] == -1).all()


def test_count_monotone_in_tau(oracle_mod):
    L = small_layer(d=128, E=32, seed=5)
    x, _ = make_tokens(30, 128, 13)
    prev = None
    for tau in np.linspace(0, 1.05, 43):
        c = oracle_mod.route(x, L.W_r, tau)["count"]
        if prev is not None:
            assert (c >= prev).all()
        prev = c
    assert (prev == 32).all()


# ---------------------------------------------------------------- expert evaluation

@pytest.mark.parametrize("perm", [False, True])
def test_all_experts_equal_dense_ffn(oracle_mod, perm):
    """Eq. (moefication_decomp): activating every expert is an identity
    transformation of the dense FFN (also after a neuron permutation)."""
    L = small_layer(d=64, E=6, seed=21, perm=perm)
    x, _ = make_tokens(9, 64, 22)
    ref = dense_ffn(x, L.W_gate, L.W_up, L.W_down)
    for tau in (1.0, 1.05):
        r, y = oracle_mod.forward(x, L.W_r, L.W_gate, L.W_up, L.W_down, tau, perm=L.perm)
        assert (r["count"] == 6).all()
        np.testing.assert_allclose(y, ref, rtol=1e-11, atol=1e-12)


def masked_dense(x, L, idx, count, scale=None):
    """Eq. (ffn) over all neurons, then zero the neurons of unkept experts
    (optionally scaling kept ones), then the down projection."""
    X = f64(x)
    H = silu(X @ f64(L.W_gate).T) * (X @ f64(L.W_up).T)
    T, d_ff = H.shape
    E = idx.shape[1]
    owner = np.empty(d_ff, np.int64)
    neurons = L.perm if L.perm is not None else np.arange(d_ff)
    owner[neurons] = np.arange(d_ff) // (d_ff // E)
    M = np.zeros((T, E))
    for t in range(T):
        M[t, idx[t, : count[t]]] = 1.0 if scale is None else scale[t, idx[t, : count[t]]]
    return (H * M[:, owner]) @ f64(L.W_down).T


@pytest.mark.parametrize("perm", [False, True])
def test_partial_selection_equals_masked_dense(oracle_mod, perm):
    L = small_layer(d=64, E=8, seed=31, perm=perm)
    x, _ = make_tokens(12, 64, 32)
    for tau in (0.0, 0.4, 0.8):
        r, y = oracle_mod.forward(x, L.W_r, L.W_gate, L.W_up, L.W_down, tau, perm=L.perm)
        np.testing.assert_allclose(y, masked_dense(x, L, r["idx"], r["count"]), rtol=1e-10,
                                   atol=1e-12)


def test_sigmoid_aggregation_equals_scaled_masked_dense(oracle_mod):
    """Eq. (moe_output): each kept expert's output scaled by sigmoid(g_e)."""
    L = small_layer(d=64, E=8, seed=41, skewed=True)
    x, it = make_tokens(10, 64, 42, temperature=True)
    fl = oracle_mod.AGG_SIGMOID
    r, y = oracle_mod.forward(x, L.W_r, L.W_gate, L.W_up, L.W_down, 0.7, flags=fl, bias=L.bias,
                              inv_temp=it)
    g = (f64(x) @ f64(L.W_r).T + L.bias) * it.astype(np.float64)[:, None]
    sig = 1.0 / (1.0 + np.exp(-g))
    np.testing.assert_allclose(y, masked_dense(x, L, r["idx"], r["count"], scale=sig),
                               rtol=1e-10, atol=1e-12)


def test_single_expert_is_dense(oracle_mod):
    L = make_layer(64, 128, 1, 51)
    x, _ = make_tokens(5, 64, 52)
    ref = dense_ffn(x, L.W_gate, L.W_up, L.W_down)
    for tau in (0.0, 0.5, 1.0):
        _, y = oracle_mod.forward(x, L.W_r, L.W_gate, L.W_up, L.W_down, tau)
        np.testing.assert_allclose(y, ref, rtol=1e-11, atol=1e-12)


def test_expert_sum_is_additive(oracle_mod):
    """y over a union of disjoint expert sets is the sum of the parts."""
    L = small_layer(d=64, E=6, seed=61)
    x, _ = make_tokens(3, 64, 62)
    A = np.array([[0, 4, -1, -1, -1, -1]] * 3, np.int32)
    B = np.array([[5, 1, 2, -1, -1, -1]] * 3, np.int32)
    AB = np.array([[2, 0, 5, 4, 1, -1]] * 3, np.int32)
    yA = oracle_mod.ffn(x, L.W_gate, L.W_up, L.W_down, A, np.full(3, 2, np.int32))
    yB = oracle_mod.ffn(x, L.W_gate, L.W_up, L.W_down, B, np.full(3, 3, np.int32))
    yAB = oracle_mod.ffn(x, L.W_gate, L.W_up, L.W_down, AB, np.full(3, 5, np.int32))
    np.testing.assert_allclose(yAB, yA + yB, rtol=1e-12, atol=1e-13)


def test_scalar_closed_form(oracle_mod):
    """One-hot token, hand-placed bf16-exact weights: every output has a
    closed form in terms of SiLU(a) b = a b / (1 + e^-a)."""
    d, E = 64, 2
    d_ff = 128 * E
    Wg = np.zeros((d_ff, d), np.float32)
    Wu = np.zeros((d_ff, d), np.float32)
    Wd = np.zeros((d, d_ff), np.float32)
    a_vals = {3: 1.5, 130: -2.0, 200: 0.25}   # neuron -> gate pre-activation
    b_vals = {3: 2.0, 130: 0.5, 200: -4.0}    # neuron -> up pre-activation
    for n in a_vals:
        Wg[n, 0] = a_vals[n]
        Wu[n, 0] = b_vals[n]
    Wd[7, 3] = 1.0
    Wd[7, 130] = 0.5
    Wd[9, 200] = -2.0
    x = np.zeros((1, d), np.float32)
    x[0, 0] = 1.0
    h = {n: a_vals[n] * b_vals[n] / (1.0 + math.exp(-a_vals[n])) for n in a_vals}
    args = [bf16_bits(v) for v in (x, Wg, Wu, Wd)]
    for sel, cnt in (([0, 1], 2), ([0, -1], 1), ([1, -1], 1)):
        y = oracle_mod.ffn(*args, np.array([sel], np.int32), np.array([cnt], np.int32))
        kept = set(sel[:cnt])
        e7 = (h[3] if 0 in kept else 0.0) + (0.5 * h[130] if 1 in kept else 0.0)
        e9 = -2.0 * h[200] if 1 in kept else 0.0
        exp = np.zeros(d)
        exp[7], exp[9] = e7, e9
        np.testing.assert_allclose(y[0], exp, rtol=1e-14, atol=1e-15)
    # sigmoid aggregation with known logits g = (2, -1)
    g = np.array([[2.0, -1.0]])
    y = oracle_mod.ffn(*args, np.array([[0, 1]], np.int32), np.array([2], np.int32),
                       flags=oracle_mod.AGG_SIGMOID, g=g)
    s0, s1 = 1 / (1 + math.exp(-2.0)), 1 / (1 + math.exp(1.0))
    assert abs(y[0, 7] - (s0 * h[3] + s1 * 0.5 * h[130])) < 1e-14
    assert abs(y[0, 9] - s1 * (-2.0) * h[200]) < 1e-14


def test_near_tie_nucleus_branch(oracle_mod):
    """Cumulative-mass ties: C_1..C_{E-1} within the band of tau (inclusive),
    C_E ignored (it is 1 and decides nothing for tau < 1), nothing at tau >= 1."""
    b = 2.0 ** -17  # exact in binary, so the band edge is exact
    cum = np.array([[0.5, 0.9 - b, 1.0],         # at the band edge: tie
                    [0.5, 0.9 - 2 * b, 1.0],     # twice the band away: no tie
                    [0.9 + b / 2, 0.95, 1.0],    # first position inside the band
                    [0.5, 0.95, 1.0]])
    assert list(oracle_mod.near_tie(cum, 0.9, band=b)) == [True, False, True, False]
    # C_E = 1 lies within the band of tau = 1 - b/2, but it is not a cut position
    cum2 = np.array([[0.5, 0.9, 1.0], [0.5, 1.0 - b, 1.0]])
    assert list(oracle_mod.near_tie(cum2, 1.0 - b / 2, band=b)) == [False, True]
    assert not oracle_mod.near_tie(cum, 1.0, band=b).any()
    assert not oracle_mod.near_tie(cum2, 1.05, band=b).any()


def test_near_tie_strict_and_rule_branches(oracle_mod):
    """Strict: tau = 1 is a cut (E - 1 kept in exact arithmetic), so masses
    within the band of 1 are ties; tau > 1 keeps all (no ties).  Top-k and
    LTE do not read C."""
    S = oracle_mod.SELECT_STRICT
    cum = np.array([[0.6, 0.999995, 1.0], [0.6, 0.99, 1.0]])
    assert list(oracle_mod.near_tie(cum, 1.0, flags=S)) == [True, False]
    assert list(oracle_mod.near_tie(cum, 0.6, flags=S)) == [True, True]
    assert not oracle_mod.near_tie(cum, 1.05, flags=S).any()
    for rule in (oracle_mod.SELECT_TOPK, oracle_mod.SELECT_LTE):
        assert not oracle_mod.near_tie(cum, 0.6, flags=rule).any()
        assert not oracle_mod.near_tie(cum, 1.0, flags=rule).any()


def test_cut_and_prefix_order_ties(oracle_mod):
    """Logit ties by position in the descending order, hand cases: a gap at
    the cut (pi_k vs pi_{k+1}), a gap inside the kept prefix, no gap, the
    band edge, nothing to cut (k = E) and logits given in expert order (the
    helpers sort them)."""
    b = 2.0 ** -17
    g = np.array([[3.0, 2.0, 2.0 - b, 0.0]])   # the tie is between ranks 2 and 3
    cases = [  # (count, tie at the cut, tie inside the prefix)
        (1, False, False), (2, True, False), (3, False, True), (4, False, True)]
    for k, cut, pre in cases:
        c = np.array([k])
        assert oracle_mod.cut_order_tie(g, c, band=b)[0] == cut, k
        assert oracle_mod.prefix_order_tie(g, c, band=b)[0] == pre, k
    # twice the band apart: no tie anywhere
    g2 = np.array([[3.0, 2.0, 2.0 - 2 * b, 0.0]])
    for k in (1, 2, 3, 4):
        assert not oracle_mod.cut_order_tie(g2, np.array([k]), band=b)[0]
        assert not oracle_mod.prefix_order_tie(g2, np.array([k]), band=b)[0]
    # the same logits in shuffled expert order, several tokens at once
    gs = np.array([[0.0, 2.0 - b, 3.0, 2.0], [2.0, 0.0, 3.0, 2.0 - b], [3.0, 2.0, 1.0, 0.0]])
    cnt = np.array([2, 3, 2])
    assert list(oracle_mod.cut_order_tie(gs, cnt, band=b)) == [True, False, False]
    assert list(oracle_mod.prefix_order_tie(gs, cnt, band=b)) == [False, True, False]
    # LTE may keep nothing: no cut, no prefix
    assert not oracle_mod.cut_order_tie(g, np.array([0]), band=b)[0]
    assert not oracle_mod.prefix_order_tie(g, np.array([0]), band=b)[0]
    # default band is the benchmark's 1e-5
    g3 = np.array([[1.0, 1.0 - 9e-6, -1.0], [1.0, 1.0 - 1.1e-5, -1.0]])
    assert list(oracle_mod.cut_order_tie(g3, np.array([1, 1]))) == [True, False]


def test_lte_tie(oracle_mod):
    """Sigmoid scores within the band of delta: logit(delta) exactly, just
    inside and just outside the band (sigmoid'(0) = 1/4), and any expert of
    the token counts."""
    d = 0.5
    inside, outside = 4 * 0.9e-6, 4 * 1.1e-6  # sigmoid(z) - 1/2 ~ z / 4
    g = np.array([[0.0, 3.0], [3.0, inside], [3.0, outside], [-outside, 5.0], [-3.0, 3.0]])
    assert list(oracle_mod.lte_tie(g, d)) == [True, True, False, False, False]
    # another delta: logit(0.9) = log 9
    g9 = np.array([[math.log(9.0), -1.0], [math.log(9.0) + 1e-3, -1.0]])
    assert list(oracle_mod.lte_tie(g9, 0.9)) == [True, False]


# ------------------------------------------- stacked-workload wiring (RMSNorm)

def test_bf16_round_matches_library_for_binary32_values(oracle_mod):
    """Every binary32 value is exact in fp64, so one rounding to bf16 must equal
    torch's binary32 -> bfloat16 conversion (round to nearest, ties to even),
    across binades, subnormals and signs."""
    import torch
    rng = np.random.default_rng(11)
    mant = rng.uniform(1.0, 2.0, 20000)
    ex = rng.integers(-140, 127, 20000)
    v = (mant * np.exp2(ex.astype(np.float64)) * rng.choice([-1.0, 1.0], 20000)).astype(np.float32)
    # exact midpoints between neighbouring bf16 values exercise the tie rule
    lo = rng.integers(0x0080, 0x7F00, 5000).astype(np.uint32)
    mids = ((lo << 16) | 0x8000).view(np.float32)
    v = np.concatenate([v, mids, -mids, np.float32([0.0, -0.0, 1.0, -2.5])])
    ref = torch.from_numpy(v).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert (oracle_mod.bf16_round(v.astype(np.float64)) == ref).all()


def test_bf16_round_is_a_single_rounding(oracle_mod):
    """Hand cases: ties go to the even significand; a value just above a tie
    (by less than binary32 resolution) rounds up, which a rounding through
    binary32 would get wrong."""
    cases = [(1.0 + 2.0 ** -8, 0x3F80), (1.0 + 3 * 2.0 ** -8, 0x3F82),
             (1.0 + 2.0 ** -8 + 2.0 ** -30, 0x3F81), (-(1.0 + 2.0 ** -8 + 2.0 ** -30), 0xBF81),
             (2.0 ** -133, 0x0001), (2.0 ** -134, 0x0000), (1.5 * 2.0 ** -134, 0x0001),
             (3.3895313892515355e38, 0x7F7F), (3.5e38, 0x7F80)]
    got = oracle_mod.bf16_round([c[0] for c in cases])
    assert [int(g) for g in got] == [c[1] for c in cases]


def test_rmsnorm_closed_forms(oracle_mod):
    # a constant row c: u = c / sqrt(c^2 + eps)
    x = np.full((2, 8), 3.0)
    x[1] = -0.25
    u, _ = oracle_mod.rmsnorm(x, 1e-5)
    assert np.allclose(u[0], 3.0 / math.sqrt(9.0 + 1e-5), rtol=1e-15, atol=0)
    assert np.allclose(u[1], -0.25 / math.sqrt(0.0625 + 1e-5), rtol=1e-15, atol=0)
    # (3, 4): mean square 12.5, so u = (0.6 sqrt 2, 0.8 sqrt 2) without eps
    u, bits = oracle_mod.rmsnorm(np.array([[3.0, 4.0]]), 0.0)
    assert np.allclose(u, [[0.6 * math.sqrt(2.0), 0.8 * math.sqrt(2.0)]], rtol=1e-15, atol=0)
    # 0.8485... lies between bf16 0.84765625 (0x3F59) and 0.8515625 (0x3F5A)
    assert bits.tolist() == [[0x3F59, 0x3F91]]


def test_rmsnorm_invariants(oracle_mod):
    rng = np.random.default_rng(5)
    x = rng.standard_normal((6, 96)) * rng.lognormal(0, 1, (6, 1))
    eps = 1e-3
    u, bits = oracle_mod.rmsnorm(x, eps)
    ms = np.mean(x * x, axis=1)
    # mean(u^2) = ms / (ms + eps); u is a positive multiple of x per row
    assert np.allclose(np.mean(u * u, axis=1), ms / (ms + eps), rtol=1e-13)
    ratio = u / x
    assert (ratio > 0).all() and np.allclose(ratio, ratio[:, :1], rtol=1e-13)
    # without eps the result is scale invariant
    u1, _ = oracle_mod.rmsnorm(x, 0.0)
    u2, _ = oracle_mod.rmsnorm(x * 37.5, 0.0)
    assert np.allclose(u1, u2, rtol=1e-13)
    # the bits are the nearest bf16 values of u
    back = bf16_to_f32(bits).astype(np.float64)
    assert (np.abs(back - u) <= np.abs(u) * 2.0 ** -8 + 1e-300).all()


# ------------------------------------------ comparison rules: top-k and LTE

def _exact_logit_layer(gvals):
    """A router whose logits for the one-hot token x = e_0 are exactly gvals
    (bf16-representable values placed in column 0 of W_r)."""
    E, d = len(gvals), 64
    W_r = np.zeros((E, d), np.float32)
    W_r[:, 0] = gvals
    x = np.zeros((1, d), np.float32)
    x[0, 0] = 1.0
    return bf16_bits(x), bf16_bits(W_r)


def test_lte_worked_cases(oracle_mod):
    """Eq. (lte_hard_set) by hand: g = (0, 1, -1, 2) gives sigmoid scores
    (0.5, 0.731, 0.269, 0.881); experts listed by descending g: 3, 1, 0, 2."""
    x, W_r = _exact_logit_layer([0.0, 1.0, -1.0, 2.0])
    for delta, kept in ((0.2, [3, 1, 0, 2]), (0.3, [3, 1, 0]), (0.5, [3, 1]),
                        (0.8, [3]), (0.9, []), (1.0, []), (0.0, [3, 1, 0, 2])):
        r = oracle_mod.route(x, W_r, delta, flags=oracle_mod.SELECT_LTE)
        k = int(r["count"][0])
        assert r["idx"][0, :k].tolist() == kept, delta
        assert (r["idx"][0, k:] == -1).all()


def test_topk_worked_cases(oracle_mod):
    x, W_r = _exact_logit_layer([0.0, 1.0, -1.0, 2.0])
    for k_arg, kept in ((2, [3, 1]), (0.4, [3]), (2.5, [3, 1, 0]), (2.49, [3, 1]),
                        (100, [3, 1, 0, 2]), (0, [3])):
        r = oracle_mod.route(x, W_r, k_arg, flags=oracle_mod.SELECT_TOPK)
        k = int(r["count"][0])
        assert r["idx"][0, :k].tolist() == kept, k_arg


def test_rules_share_the_order(oracle_mod):
    """Every rule keeps a prefix of the same order pi; top-k with the nucleus
    count reproduces the nucleus selection; LTE counts fall as delta rises."""
    L = small_layer(d=128, E=10, seed=21)
    x, _ = make_tokens(40, 128, 22)
    nuc = oracle_mod.route(x, L.W_r, 0.6)
    full = oracle_mod.route(x, L.W_r, 1.0)
    for t in range(40):
        k = int(nuc["count"][t])
        top = oracle_mod.route(x[t:t + 1], L.W_r, float(k), flags=oracle_mod.SELECT_TOPK)
        assert top["idx"][0, :k].tolist() == nuc["idx"][t, :k].tolist()
    prev = None
    for delta in (0.05, 0.2, 0.5, 0.8, 0.95, 0.999):
        r = oracle_mod.route(x, L.W_r, delta, flags=oracle_mod.SELECT_LTE)
        for t in range(40):
            k = int(r["count"][t])
            assert r["idx"][t, :k].tolist() == full["idx"][t, :k].tolist()
            s = 1.0 / (1.0 + np.exp(-r["g"][t]))
            assert k == int((s > delta).sum())
        if prev is not None:
            assert (r["count"] <= prev).all()
        prev = r["count"]


# ------------------------------------------------- routing regularisers (Sec. 3.2)
def _sig(v):
    return 1.0 / (1.0 + np.exp(-v))


def test_router_loss_uniform_closed_form(oracle_mod):
    """Equal logits: p = 1/E, so L_ent = log E (eps = 0), L_bal = 1, L_gate =
    sigmoid(c); uniform routing is a stationary point of L_ent and L_bal, so
    only the gate term's gradient sigmoid'(c) / (B E) is left."""
    for B, E, c in [(1, 1, 0.0), (3, 8, 0.7), (16, 112, -2.5), (5, 256, 3.0)]:
        g = np.full((B, E), c)
        for eta, lam, gam in [(1.0, 0.0, 0.0), (0.3, 2.0, 0.5)]:
            L, dg = oracle_mod.router_loss(g, eps=0.0, eta=eta, lam=lam, gamma=gam)
            s = _sig(c)
            want = [math.log(E), 1.0, s]
            np.testing.assert_allclose(L[:3], want, rtol=1e-13, atol=1e-15)
            assert L[3] == pytest.approx(eta * want[0] + lam * want[1] + gam * want[2], rel=1e-13)
            np.testing.assert_allclose(dg, gam * s * (1 - s) / (B * E), rtol=1e-9, atol=1e-17)


def test_router_loss_two_experts_is_binary_entropy(oracle_mod):
    """E = 2: softmax of two logits is the logistic function of their
    difference, so L_ent is the mean binary entropy (scipy.stats.entropy) and
    m_0 the mean of sigmoid(g_0 - g_1)."""
    from scipy.stats import entropy
    rng = np.random.default_rng(11)
    g = rng.normal(0, 2, (9, 2))
    L, _ = oracle_mod.router_loss(g, eps=0.0, grad=False)
    q = _sig(g[:, 0] - g[:, 1])
    ent = np.mean([entropy([a, 1 - a]) for a in q])
    m0 = q.mean()
    assert L[0] == pytest.approx(ent, rel=1e-12)
    assert L[1] == pytest.approx(2 * (m0 ** 2 + (1 - m0) ** 2), rel=1e-12)
    assert L[2] == pytest.approx(_sig(g).mean(), rel=1e-12)


def test_router_loss_cyclic_rows_are_balanced(oracle_mod):
    """B = E rows that are the E cyclic shifts of one logit vector: every
    expert receives the same total mass, so L_bal = 1 exactly, and every row
    has the entropy of the first (scipy.stats.entropy of scipy's softmax)."""
    from scipy.stats import entropy
    rng = np.random.default_rng(5)
    E = 13
    v = rng.normal(0, 3, E)
    g = np.stack([np.roll(v, s) for s in range(E)])
    L, _ = oracle_mod.router_loss(g, eps=0.0, grad=False)
    assert L[1] == pytest.approx(1.0, rel=1e-12)
    assert L[0] == pytest.approx(entropy(sp_softmax(v)), rel=1e-12)


def test_router_loss_collapse_and_bounds(oracle_mod):
    """Sum_j m_j = 1 gives 1 <= L_bal <= E (equality only for uniform m, or
    all mass on one expert); L_ent lies in [0, log E] for eps = 0, decreases
    as eps grows, and a one-hot batch gives L_ent = 0, L_bal = E."""
    rng = np.random.default_rng(8)
    for E in (2, 7, 64):
        g = rng.normal(0, 4, (20, E))
        L0, _ = oracle_mod.router_loss(g, eps=0.0, grad=False)
        L1, _ = oracle_mod.router_loss(g, eps=1e-2, grad=False)
        assert 1.0 < L0[1] < E
        assert 0.0 < L0[0] < math.log(E)
        assert L1[0] < L0[0] and L1[1] == L0[1]
        hot = np.full((6, E), -1e4)
        hot[:, E - 1] = 0.0          # p = e_{E-1} exactly in fp64 (exp underflows)
        L, dg = oracle_mod.router_loss(hot, eps=0.0, eta=1.0, lam=0.0)
        assert L[0] == 0.0 and L[1] == pytest.approx(E, rel=1e-15)
        assert np.isfinite(dg).all()


def test_router_loss_batch_normalisation(oracle_mod):
    """L_ent, L_bal and L_gate are batch means: a batch repeated twice has the
    same losses, and its gradient is half the single batch's per row."""
    rng = np.random.default_rng(2)
    g = rng.normal(0, 1.5, (7, 10))
    kw = dict(eps=1e-6, eta=0.7, lam=1.3, gamma=0.4)
    L1, d1 = oracle_mod.router_loss(g, **kw)
    L2, d2 = oracle_mod.router_loss(np.vstack([g, g]), **kw)
    np.testing.assert_allclose(L2, L1, rtol=1e-13)
    np.testing.assert_allclose(d2[:7], d1 / 2, rtol=1e-11, atol=1e-18)
    np.testing.assert_allclose(d2[7:], d1 / 2, rtol=1e-11, atol=1e-18)


def test_router_loss_permutation_equivariance(oracle_mod):
    """Reordering tokens or relabelling experts leaves the losses unchanged
    and moves the gradient's rows or columns with them."""
    rng = np.random.default_rng(4)
    g = rng.normal(0, 2, (6, 9))
    kw = dict(eps=1e-4, eta=0.5, lam=2.0, gamma=0.3)
    L, d = oracle_mod.router_loss(g, **kw)
    r, c = rng.permutation(6), rng.permutation(9)
    Lp, dp = oracle_mod.router_loss(g[r][:, c], **kw)
    np.testing.assert_allclose(Lp, L, rtol=1e-13)
    np.testing.assert_allclose(dp, d[r][:, c], rtol=1e-11, atol=1e-18)


def test_router_loss_gradient_rows_sum_to_zero(oracle_mod):
    """Softmax is unchanged by adding a constant to a row's logits, so the
    gradient of L_ent + L_bal sums to zero over each row."""
    rng = np.random.default_rng(6)
    g = rng.normal(0, 3, (8, 33))
    _, d = oracle_mod.router_loss(g, eps=1e-3, eta=0.8, lam=1.7, gamma=0.0)
    assert np.abs(d.sum(axis=1)).max() < 1e-15 * 33 + 1e-17
    assert np.abs(d).max() > 1e-4


@pytest.mark.parametrize("coef", [(1, 0, 0), (0, 1, 0), (0, 0, 1), (0.6, 1.4, 0.9)])
def test_router_loss_gradient_finite_differences(oracle_mod, coef):
    """dL/dg against central differences of the oracle's own forward loss,
    one term at a time and all together, with eps large enough that the
    eps-dependent part of d[p log(p + eps)]/dp matters."""
    eta, lam, gam = coef
    rng = np.random.default_rng(9)
    B, E, eps = 4, 6, 5e-2
    g = rng.normal(0, 1.5, (B, E))
    _, d = oracle_mod.router_loss(g, eps=eps, eta=eta, lam=lam, gamma=gam)
    h = 1e-5
    fd = np.empty_like(g)
    for i in range(B):
        for j in range(E):
            gp, gm = g.copy(), g.copy()
            gp[i, j] += h
            gm[i, j] -= h
            Lp, _ = oracle_mod.router_loss(gp, eps=eps, eta=eta, lam=lam, gamma=gam, grad=False)
            Lm, _ = oracle_mod.router_loss(gm, eps=eps, eta=eta, lam=lam, gamma=gam, grad=False)
            fd[i, j] = (Lp[3] - Lm[3]) / (2 * h)
    np.testing.assert_allclose(d, fd, rtol=1e-6, atol=1e-10)


# ------------------------------------------- non-gated GELU MLP variant (Sec. 2.1)
def test_gelu_matches_torch_tanh_form(oracle_mod):
    """The oracle's GELU against torch's tanh-form GELU in float64, and the
    identity GELU(a) - GELU(-a) = a (the tanh term is odd)."""
    import torch
    a = np.concatenate([np.linspace(-12, 12, 401), [0.0, 1e-8, -1e-8, 30.0, -30.0]])
    ref = torch.nn.functional.gelu(torch.from_numpy(a), approximate="tanh").numpy()
    got = oracle_mod.gelu(a)
    # 1 + tanh(u) cancels for large negative a: absolute error ~ |a| ulp there
    np.testing.assert_allclose(got, ref, rtol=1e-14, atol=1e-14)
    np.testing.assert_allclose(got - oracle_mod.gelu(-a), a, rtol=1e-13, atol=1e-15)
    assert oracle_mod.gelu(np.array([0.0]))[0] == 0.0


def dense_mlp(x, L):
    """GELU(x W_fc^T + b_fc) W_proj^T + b_proj, numpy float64 with torch's
    GELU, no experts."""
    import torch
    X, Wf, Wp = f64(x), f64(L.W_fc), f64(L.W_proj)
    a = X @ Wf.T + L.b_fc.astype(np.float64)
    h = torch.nn.functional.gelu(torch.from_numpy(a), approximate="tanh").numpy()
    return h @ Wp.T + L.b_proj.astype(np.float64)


def all_experts(T, E):
    return np.tile(np.arange(E, dtype=np.int32), (T, 1)), np.full(T, E, np.int32)


@pytest.mark.parametrize("perm", [False, True])
def test_mlp_all_experts_equal_dense(oracle_mod, perm):
    """Eq. (moefication_decomp) for the non-gated MLP: all experts (in any
    order, after any neuron permutation) give the dense MLP, biases included."""
    from paper_2605_28283_amd.workloads import make_mlp_layer
    L = make_mlp_layer(64, 128 * 5, 5, 7, perm=perm)
    x, _ = make_tokens(6, 64, 8)
    idx, cnt = all_experts(6, 5)
    idx = idx[:, ::-1].copy()
    y = oracle_mod.mlp(x, L.W_fc, L.b_fc, L.W_proj, L.b_proj, idx, cnt, perm=L.perm)
    np.testing.assert_allclose(y, dense_mlp(x, L), rtol=1e-11, atol=1e-13)


def test_mlp_partial_selection_and_bias_once(oracle_mod):
    """A partial selection equals the dense MLP with the other neurons' h set
    to zero; b_proj is added once (a token that keeps no expert gets
    y = b_proj); disjoint selections add up after removing b_proj; sigmoid
    aggregation scales each expert's block."""
    import torch
    from paper_2605_28283_amd.workloads import make_mlp_layer
    E, d = 6, 64
    L = make_mlp_layer(d, 128 * E, E, 9)
    x, _ = make_tokens(3, d, 10)
    X = f64(x)
    a = X @ f64(L.W_fc).T + L.b_fc.astype(np.float64)
    h = torch.nn.functional.gelu(torch.from_numpy(a), approximate="tanh").numpy()
    sel = [[4, 1], [0], []]
    idx = np.full((3, E), -1, np.int32)
    cnt = np.array([len(s) for s in sel], np.int32)
    for t, s in enumerate(sel):
        idx[t, :len(s)] = s
    y = oracle_mod.mlp(x, L.W_fc, L.b_fc, L.W_proj, L.b_proj, idx, cnt)
    g = np.random.default_rng(0).normal(0, 2, (3, E))
    ys = oracle_mod.mlp(x, L.W_fc, L.b_fc, L.W_proj, L.b_proj, idx, cnt, flags=2, g=g)
    for t, s in enumerate(sel):
        mask = np.zeros(128 * E)
        scl = np.zeros(128 * E)
        for e in s:
            mask[128 * e:128 * e + 128] = 1.0
            scl[128 * e:128 * e + 128] = 1.0 / (1.0 + np.exp(-g[t, e]))
        ref = (h[t] * mask) @ f64(L.W_proj).T + L.b_proj
        np.testing.assert_allclose(y[t], ref, rtol=1e-11, atol=1e-13)
        np.testing.assert_allclose(ys[t], (h[t] * scl) @ f64(L.W_proj).T + L.b_proj,
                                   rtol=1e-11, atol=1e-13)
    np.testing.assert_array_equal(y[2], L.b_proj.astype(np.float64))
    i1 = np.array([[4, -1, -1, -1, -1, -1]], np.int32)
    i2 = np.array([[1, -1, -1, -1, -1, -1]], np.int32)
    one = np.array([1], np.int32)
    y1 = oracle_mod.mlp(x[:1], L.W_fc, L.b_fc, L.W_proj, L.b_proj, i1, one)
    y2 = oracle_mod.mlp(x[:1], L.W_fc, L.b_fc, L.W_proj, L.b_proj, i2, one)
    np.testing.assert_allclose((y1 - L.b_proj) + (y2 - L.b_proj), y[:1] - L.b_proj,
                               rtol=1e-11, atol=1e-13)


def test_mlp_scalar_closed_form(oracle_mod):
    """One-hot weights: y_i = b_proj[i] + W_proj[i, n] GELU(x_j W_fc[n, j] +
    b_fc[n]) for the single live neuron n, written out by hand."""
    from paper_2605_28283_amd.workloads import MlpLayer, bf16_bits
    d, E = 64, 1
    d_ff = 128
    W_r = bf16_bits(np.zeros((E, d), np.float32))
    W_fc = np.zeros((d_ff, d), np.float32)
    W_proj = np.zeros((d, d_ff), np.float32)
    W_fc[37, 5] = 1.5
    W_proj[11, 37] = -0.75
    b_fc = np.zeros(d_ff, np.float32)
    b_fc[37] = 0.25
    b_proj = np.zeros(d, np.float32)
    b_proj[3] = 0.5
    L = MlpLayer(d, d_ff, E, W_r, bf16_bits(W_fc), b_fc, bf16_bits(W_proj), b_proj)
    xv = np.zeros((1, d), np.float32)
    xv[0, 5] = 2.0
    y = oracle_mod.mlp(bf16_bits(xv), L.W_fc, L.b_fc, L.W_proj, L.b_proj,
                       np.zeros((1, 1), np.int32), np.ones(1, np.int32))
    a = 2.0 * 1.5 + 0.25
    gelu_a = 0.5 * a * (1 + math.tanh(math.sqrt(2 / math.pi) * (a + 0.044715 * a ** 3)))
    want = np.zeros(d)
    want[3] = 0.5
    want[11] = -0.75 * gelu_a
    np.testing.assert_allclose(y[0], want, rtol=1e-14, atol=1e-15)


# ----------------------------------------- balanced k-means (MoEfication, Sec. 2.2)
def _balanced_splits(n, k):
    """Every assignment of n labelled rows to k labelled clusters of n/k rows."""
    m = n // k

    def rec(rest, j):
        if j == k - 1:
            yield {j: rest}
            return
        for c in itertools.combinations(rest, m):
            left = tuple(r for r in rest if r not in c)
            for tail in rec(left, j + 1):
                tail = dict(tail)
                tail[j] = c
                yield tail
    for split in rec(tuple(range(n)), 0):
        a = np.empty(n, np.int64)
        for j, rows in split.items():
            a[list(rows)] = j
        yield a


@pytest.mark.parametrize("n,k,seed", [(8, 2, 0), (9, 3, 1), (8, 4, 2), (12, 3, 3)])
def test_kmeans_assignment_brute_force(n, k, seed):
    """The balanced assignment's cost is the minimum over every balanced
    assignment (enumerated), and the assignment is balanced."""
    from oracle import kmeans
    rng = np.random.default_rng(seed)
    X = rng.normal(0, 1, (n, 3))
    mu = rng.normal(0, 1, (k, 3))
    a, cost = kmeans.balanced_assign(X, mu)
    assert (np.bincount(a, minlength=k) == n // k).all()
    S = ((X[:, None, :] - mu[None]) ** 2).sum(-1)
    best = min(S[np.arange(n), b].sum() for b in _balanced_splits(n, k))
    assert cost == pytest.approx(best, rel=1e-12)


def test_kmeans_planted_clusters_recovered():
    """Rows scattered tightly around k far-apart centres, m per centre, in a
    shuffled order: one iteration from one row of each group returns the
    planted groups, their means as centroids and Pi listing them."""
    from oracle import kmeans
    rng = np.random.default_rng(4)
    k, m, D = 6, 8, 5
    centres = rng.normal(0, 10, (k, D))
    X = np.repeat(centres, m, axis=0) + rng.normal(0, 0.01, (k * m, D))
    order = rng.permutation(k * m)
    X = X[order]
    group = np.repeat(np.arange(k), m)[order]
    init = np.stack([X[np.nonzero(group == j)[0][0]] for j in range(k)])
    r = kmeans.balanced_kmeans(X, init, 1)
    np.testing.assert_array_equal(r["assign"], group)
    for j in range(k):
        np.testing.assert_allclose(r["centroids"][j], X[group == j].mean(0), rtol=1e-12)
        np.testing.assert_array_equal(r["perm"][j * m:(j + 1) * m], np.nonzero(group == j)[0])


def test_kmeans_unconstrained_when_already_balanced():
    """If every row's nearest centroid already gives m rows per cluster, the
    balanced assignment is the nearest-centroid assignment."""
    from oracle import kmeans
    rng = np.random.default_rng(5)
    k, m = 4, 6
    mu = np.eye(k, 4) * 20
    X = np.repeat(mu, m, axis=0) + rng.normal(0, 1, (k * m, 4))
    a, _ = kmeans.balanced_assign(X, mu)
    near = np.argmin(((X[:, None] - mu[None]) ** 2).sum(-1), axis=1)
    assert (np.bincount(near, minlength=k) == m).all()
    np.testing.assert_array_equal(a, near)


def test_kmeans_objective_monotone_and_perm_valid():
    """Lloyd's steps never increase the objective (the assignment is optimal
    for fixed centroids, the means for a fixed assignment); Pi is a
    permutation whose blocks are the clusters, ascending."""
    from oracle import kmeans
    rng = np.random.default_rng(6)
    n, k, D = 96, 8, 7
    X = rng.normal(0, 1, (n, D))
    init = X[rng.choice(n, k, replace=False)]
    r = kmeans.balanced_kmeans(X, init, 6)
    assert (np.diff(r["objective"]) <= 1e-9 * r["objective"][0]).all()
    p = r["perm"]
    assert sorted(p.tolist()) == list(range(n))
    m = n // k
    for j in range(k):
        blk = p[j * m:(j + 1) * m]
        assert (r["assign"][blk] == j).all() and (np.diff(blk) > 0).all()
    # the objective after the last update is the cost of the last assignment
    # evaluated at the updated centroids, which is no larger
    last = ((X - r["centroids"][r["assign"]]) ** 2).sum()
    assert last <= r["objective"][-1] + 1e-9
