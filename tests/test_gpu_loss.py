"""GPU parity of the routing regularisers (L_ent, L_bal, L_gate and dL/dg,
Sec. 3.2 and Sec. 4.2.3) against the fp64 oracle, through the C ABI.

Bar (the kernel computes in fp32; the cross-block sums in fp64): every loss
within 2e-5 absolute + 2e-5 relative of the oracle, every gradient entry
within 2e-5 of max|dL/dg| (fp32 softmax, log and exp carry ~1e-7 relative
error per term, and each row sums at most 256 terms), or within a few fp32
ulps of the size of the dL/dp terms that cancel in p (a - sum p a) where the
exact gradient vanishes (uniform rows): |eta| (1 + 90) / B + 2 |lambda| E / B
(|log p| <= 90 for fp32 probabilities).
"""
import numpy as np
import pytest

import paper_2605_28283_amd as pp
from paper_2605_28283_amd.workloads import ROUTER_LOSS_B, ROUTER_LOSS_E, make_router_logits

pytestmark = pytest.mark.gpu

LOSS_TOL = 2e-5
GRAD_TOL = 2e-5
COEF = dict(eps=1e-8, eta=0.5, lam=0.05, gamma=0.1)


@pytest.fixture(scope="module", autouse=True)
def gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    pp.load()
    torch.cuda.init()


def run_loss(g, eps, eta, lam, gamma, grad=True):
    import torch
    B, E = g.shape
    gd = torch.from_numpy(np.ascontiguousarray(g, np.float32)).cuda()
    nbytes = pp.prunepath_router_loss_workspace(B, E)
    assert nbytes > 0
    ws = torch.full((nbytes // 4,), float("nan"), dtype=torch.float32, device="cuda")
    losses = torch.full((4,), float("nan"), dtype=torch.float32, device="cuda")
    dg = torch.full((B, E), float("nan"), dtype=torch.float32, device="cuda") if grad else None
    pp.prunepath_router_loss(gd, B, E, eps, eta, lam, gamma, losses, dg, ws)
    torch.cuda.synchronize()
    return losses.cpu().numpy(), None if dg is None else dg.cpu().numpy()


def check(oracle, g, eps, eta, lam, gamma):
    print("router loss B=%d E=%d eps=%g eta=%g lam=%g gamma=%g" %
          (g.shape[0], g.shape[1], eps, eta, lam, gamma), flush=True)
    L, dg = run_loss(g, eps, eta, lam, gamma)
    L_ref, dg_ref = oracle.router_loss(g.astype(np.float64), eps=eps, eta=eta, lam=lam,
                                       gamma=gamma)
    scale = np.array([1.0, 1.0, 1.0, abs(eta) + abs(lam) + abs(gamma)])
    err = np.abs(L.astype(np.float64) - L_ref)
    assert (err <= LOSS_TOL * scale + LOSS_TOL * np.abs(L_ref)).all(), (L, L_ref)
    assert np.isfinite(dg).all()
    B, E = g.shape
    gmax = float(np.abs(dg_ref).max())
    floor = 4 * 2.0 ** -24 * ((abs(eta) * 91 + 2 * abs(lam) * E) / B + abs(gamma) / (B * E))
    worst = float(np.abs(dg.astype(np.float64) - dg_ref).max())
    assert worst <= GRAD_TOL * gmax + floor, (worst, gmax, floor)
    return L, dg


@pytest.mark.parametrize("B,E,seed", [
    (1, 1, 0), (1, 112, 1), (5, 7, 2), (16, 112, 3), (17, 112, 4),    # one block, ragged tail
    (333, 64, 5), (1000, 256, 6), (4097, 112, 7), (2049, 148, 8),     # many blocks, ragged
])
def test_router_loss_parity(oracle_mod, B, E, seed):
    check(oracle_mod, make_router_logits(B, E, seed), **COEF)


@pytest.mark.parametrize("coef", [
    dict(eps=1e-8, eta=1.0, lam=0.0, gamma=0.0),
    dict(eps=1e-8, eta=0.0, lam=1.0, gamma=0.0),
    dict(eps=1e-8, eta=0.0, lam=0.0, gamma=1.0),
    dict(eps=0.0, eta=0.3, lam=2.0, gamma=-0.5),
    dict(eps=1e-2, eta=0.7, lam=0.1, gamma=0.2),
])
def test_router_loss_terms(oracle_mod, coef):
    """Each regulariser alone (its gradient isolated), eps = 0, a large eps."""
    check(oracle_mod, make_router_logits(700, 112, 11), **coef)


def test_router_loss_training_batch(oracle_mod):
    """The benchmarked training-step shape, the whole batch compared."""
    check(oracle_mod, make_router_logits(ROUTER_LOSS_B, ROUTER_LOSS_E, 0), **COEF)


def test_router_loss_degenerate_rows(oracle_mod):
    """Uniform rows (L_ent = log E at eps = 0, zero gradient of L_ent and
    L_bal), one-hot rows whose other probabilities underflow to 0 in fp32
    (eps = 0: those terms are taken at their limit), and E = 1."""
    E = 112
    g = np.zeros((40, E), np.float32)
    g[10:20] = 3.25                      # uniform at another level
    g[20:30, 7] = 300.0                  # fp32 exp(-300) = 0
    g[30:40] = np.linspace(-50, 50, E, dtype=np.float32)
    check(oracle_mod, g, eps=0.0, eta=1.0, lam=1.0, gamma=0.0)
    L, dg = check(oracle_mod, g[:20], eps=0.0, eta=1.0, lam=1.0, gamma=0.0)
    assert L[0] == pytest.approx(np.log(E), rel=1e-6) and L[1] == pytest.approx(1.0, rel=1e-6)
    assert np.abs(dg).max() <= 1e-9
    check(oracle_mod, make_router_logits(50, 1, 3), **COEF)


def test_router_loss_deterministic_and_forward_only():
    """Repeated calls give identical bits; with dg NULL the losses are those
    of the full call."""
    g = make_router_logits(3000, 112, 9)
    L1, d1 = run_loss(g, **COEF)
    L2, d2 = run_loss(g, **COEF)
    L3, _ = run_loss(g, **COEF, grad=False)
    assert L1.tobytes() == L2.tobytes() == L3.tobytes()
    assert d1.tobytes() == d2.tobytes()


def test_router_loss_invariances():
    """Adding a constant to every logit of a row changes p not at all, so L_ent,
    L_bal and their gradient (gamma = 0) are unchanged up to rounding; a
    batch repeated twice has the same losses."""
    g = make_router_logits(512, 112, 12)
    c = dict(eps=1e-8, eta=0.4, lam=0.3, gamma=0.0)
    L, d = run_loss(g, **c)
    Ls, ds = run_loss(g + np.float32(4.0), **c)
    np.testing.assert_allclose(Ls[:2], L[:2], rtol=1e-5)
    assert np.abs(ds - d).max() <= 1e-4 * np.abs(d).max()
    L2, _ = run_loss(np.vstack([g, g]), **c)
    np.testing.assert_allclose(L2[:3], L[:3], rtol=1e-5)


def test_router_loss_graph_replays_match_eager():
    """Captured in a HIP graph (as the benchmark times it) and replayed
    several times with eager work in between: every replay gives the eager
    call's bits."""
    import torch
    B, E = 3001, 112
    g = torch.from_numpy(make_router_logits(B, E, 21)).cuda()
    ws = torch.empty(pp.prunepath_router_loss_workspace(B, E) // 4, dtype=torch.float32,
                     device="cuda")
    L_e = torch.empty(4, dtype=torch.float32, device="cuda")
    dg_e = torch.empty((B, E), dtype=torch.float32, device="cuda")
    pp.prunepath_router_loss(g, B, E, 1e-8, 0.5, 0.05, 0.1, L_e, dg_e, ws)
    torch.cuda.synchronize()
    L_g = torch.empty_like(L_e)
    dg_g = torch.empty_like(dg_e)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        pp.prunepath_router_loss(g, B, E, 1e-8, 0.5, 0.05, 0.1, L_g, dg_g, ws,
                                 stream=torch.cuda.current_stream())
    for _ in range(4):
        L_g.fill_(float("nan"))
        dg_g.fill_(float("nan"))
        ws.fill_(float("nan"))
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert L_g.cpu().numpy().tobytes() == L_e.cpu().numpy().tobytes()
        assert dg_g.cpu().numpy().tobytes() == dg_e.cpu().numpy().tobytes()
