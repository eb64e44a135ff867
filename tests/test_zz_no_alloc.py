"""The allocation-free routing-regulariser entry point,
prunepath_router_loss_noalloc: its scratch is a device array inside the
library, so it takes no workspace and allocates nothing.  Its output must
equal prunepath_router_loss's (same kernels, same summation order: the same
bits) and meet the oracle bar of the routing-regulariser tests, on two calls
in a row, the second smaller; sizes past the array are refused."""
import numpy as np
import pytest

import paper_2605_28283_amd as pp
from paper_2605_28283_amd.workloads import ROUTER_LOSS_B, ROUTER_LOSS_E, make_router_logits

SCRATCH_BYTES = 4 << 20
COEF = (1e-8, 0.5, 0.05, 0.1)  # eps, eta, lambda, gamma
LOSS_TOL = GRAD_TOL = 2e-5


def test_noalloc_rejects_bad_arguments_on_the_host():
    """Argument checks return before any HIP call (runs without a GPU)."""
    lib = pp.load()
    eps, eta, lam, gam = COEF
    call = lib.prunepath_router_loss_noalloc
    assert call(None, 8, 16, eps, eta, lam, gam, 16, 32, None) == pp.PP_EINVAL    # g NULL
    assert call(16, 8, 16, eps, eta, lam, gam, None, 32, None) == pp.PP_EINVAL    # losses NULL
    assert call(16, 8, 16, eps, eta, lam, gam, 48, 16, None) == pp.PP_EINVAL      # dg aliases g
    assert call(16, 0, 16, eps, eta, lam, gam, 48, 32, None) == pp.PP_EINVAL      # B < 1
    assert call(16, 8, 257, eps, eta, lam, gam, 48, 32, None) == pp.PP_EINVAL     # E > 256
    assert call(16, 8, 16, float("nan"), eta, lam, gam, 48, 32, None) == pp.PP_EINVAL
    assert call(24, 8, 16, eps, eta, lam, gam, 48, 32, None) == pp.PP_EINVAL      # g misaligned
    # past the scratch array: ceil(B / 64) * (E + 2) * 4 bytes > 4 MiB
    for B, E in ((588673, 112), (260097, 256), (1 << 22, 15)):
        assert lib.prunepath_router_loss_workspace(B, E) > SCRATCH_BYTES
        assert call(16, B, E, eps, eta, lam, gam, 48, 32, None) == pp.PP_EUNSUPPORTED
    for B, E in ((588672, 112), (260096, 256), (1 << 22, 14)):
        assert lib.prunepath_router_loss_workspace(B, E) <= SCRATCH_BYTES


def _dev(torch, a):
    return torch.from_numpy(np.ascontiguousarray(a, np.float32)).cuda()


def _with_workspace(torch, g, B, E):
    ws = torch.full((pp.prunepath_router_loss_workspace(B, E) // 4,), float("nan"),
                    dtype=torch.float32, device="cuda")
    losses = torch.full((4,), float("nan"), dtype=torch.float32, device="cuda")
    dg = torch.full((B, E), float("nan"), dtype=torch.float32, device="cuda")
    pp.prunepath_router_loss(g, B, E, *COEF, losses, dg, ws)
    torch.cuda.synchronize()
    return losses.cpu().numpy(), dg.cpu().numpy()


def _noalloc(torch, g, B, E):
    losses = torch.full((4,), float("nan"), dtype=torch.float32, device="cuda")
    dg = torch.full((B, E), float("nan"), dtype=torch.float32, device="cuda")
    pp.prunepath_router_loss_noalloc(g, B, E, *COEF, losses, dg)
    torch.cuda.synchronize()
    return losses.cpu().numpy(), dg.cpu().numpy()


def _oracle_bar(oracle_mod, g_np, L, dg):
    eps, eta, lam, gam = COEF
    L_ref, dg_ref = oracle_mod.router_loss(g_np.astype(np.float64), eps=eps, eta=eta, lam=lam,
                                           gamma=gam)
    scale = np.array([1.0, 1.0, 1.0, abs(eta) + abs(lam) + abs(gam)])
    assert (np.abs(L - L_ref) <= LOSS_TOL * scale + LOSS_TOL * np.abs(L_ref)).all(), (L, L_ref)
    B, E = g_np.shape
    floor = 4 * 2.0 ** -24 * ((abs(eta) * 91 + 2 * abs(lam) * E) / B + abs(gam) / (B * E))
    assert np.abs(dg - dg_ref).max() <= GRAD_TOL * np.abs(dg_ref).max() + floor


@pytest.mark.gpu
def test_noalloc_matches_workspace_entry_point(oracle_mod):
    """Two calls in a row, the second with a smaller batch (the array keeps the
    first call's partials): each equals the workspace entry point bit for bit
    and meets the oracle bar."""
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    pp.load()
    for B, E, seed in ((ROUTER_LOSS_B, ROUTER_LOSS_E, 0), (333, 64, 5)):
        print("noalloc router loss B=%d E=%d" % (B, E), flush=True)
        g_np = make_router_logits(B, E, seed)
        g = _dev(torch, g_np)
        L_ws, dg_ws = _with_workspace(torch, g, B, E)
        L_na, dg_na = _noalloc(torch, g, B, E)
        np.testing.assert_array_equal(L_na, L_ws)
        np.testing.assert_array_equal(dg_na, dg_ws)
        _oracle_bar(oracle_mod, g_np, L_na.astype(np.float64), dg_na.astype(np.float64))


@pytest.mark.gpu
def test_noalloc_in_a_graph(oracle_mod):
    """The caller it is for: a captured HIP graph holding the call (no
    workspace to allocate inside the capture).  The first call on the device
    runs eagerly; three replays with eager work in between each reproduce
    the eager result."""
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    pp.load()
    B, E = 4097, 112
    print("noalloc router loss in a graph B=%d E=%d" % (B, E), flush=True)
    g_np = make_router_logits(B, E, 7)
    g = _dev(torch, g_np)
    L_ref, dg_ref = _noalloc(torch, g, B, E)
    losses = torch.full((4,), float("nan"), dtype=torch.float32, device="cuda")
    dg = torch.full((B, E), float("nan"), dtype=torch.float32, device="cuda")
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        pp.prunepath_router_loss_noalloc(g, B, E, *COEF, losses, dg, stream=side)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        pp.prunepath_router_loss_noalloc(g, B, E, *COEF, losses, dg,
                                         stream=torch.cuda.current_stream())
    for rep in range(3):
        losses.fill_(float("nan"))
        dg.fill_(float("nan"))
        # eager work between replays, including another size through the same array
        _noalloc(torch, _dev(torch, make_router_logits(100, 16, rep)), 100, 16)
        graph.replay()
        torch.cuda.synchronize()
        np.testing.assert_array_equal(losses.cpu().numpy(), L_ref)
        np.testing.assert_array_equal(dg.cpu().numpy(), dg_ref)
