"""GPU parity of the stacked-layer decode workload: the residual + RMSNorm
kernel against the oracle, and the 32-layer LLaMA-3-8B-shaped stack (T=16,
tau=0.8) checked layer by layer, teacher-forced: the oracle's layer l takes
the GPU's own input of that layer (one near-tie flip would otherwise change
every later layer).  The stack runs in the same HIP-graph launch
configuration the benchmark times, and every replay must reproduce the eager
step bit for bit.
"""
import numpy as np
import pytest

import paper_2605_28283_amd as pp
from paper_2605_28283_amd.stack import DecodeStack
from paper_2605_28283_amd.workloads import (WORKLOADS, Layer, bf16_to_f32, make_layer_device,
                                            stack_layer_seed, workload_tokens)
from gpu_helpers import check_output, check_selection, full_size_cap

pytestmark = pytest.mark.gpu

MID_BAND = 2.0 ** -19   # relative distance to a bf16 rounding midpoint treated as a tie


@pytest.fixture(scope="module", autouse=True)
def gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    pp.load()
    torch.cuda.init()


def check_bf16_rounding(u_ref, bits_ref, bits_gpu):
    """GPU bf16 bits equal the oracle's nearest-even rounding of the fp64
    value, except where that value lies within MID_BAND of the midpoint
    between two bf16 neighbours; there the other neighbour is accepted.
    Returns the number of such ties."""
    bits_gpu = np.asarray(bits_gpu).view(np.uint16)
    diff = bits_gpu != bits_ref
    if not diff.any():
        return 0
    vr = bf16_to_f32(bits_ref[diff]).astype(np.float64)
    vg = bf16_to_f32(bits_gpu[diff]).astype(np.float64)
    v = u_ref[diff]
    neighbours = np.abs(bits_gpu[diff].astype(np.int64) - bits_ref[diff].astype(np.int64)) == 1
    near_mid = np.abs(v - 0.5 * (vr + vg)) <= MID_BAND * np.abs(v)
    ok = neighbours & near_mid
    assert ok.all(), "bf16 rounding mismatch at %d entries" % int((~ok).sum())
    return int(diff.sum())


@pytest.mark.parametrize("T,d", [(1, 4), (3, 64), (5, 1000), (16, 4096), (7, 8192)])
@pytest.mark.parametrize("with_y", [False, True])
def test_residual_rmsnorm(oracle_mod, T, d, with_y):
    import torch
    rng = np.random.default_rng(T * 1000 + d)
    x = (rng.standard_normal((T, d)) * rng.lognormal(0, 1, (T, 1))).astype(np.float32)
    y = rng.standard_normal((T, d)).astype(np.float32) * 0.3
    xd = torch.from_numpy(x).cuda()
    yd = torch.from_numpy(y).cuda() if with_y else None
    xo = torch.full((T, d), float("nan"), device="cuda")
    u = torch.full((T, d), -1, dtype=torch.int16, device="cuda")
    pp.prunepath_residual_rmsnorm(xd, yd, xo, T, d, 1e-5, u)
    torch.cuda.synchronize()
    xs = x + y if with_y else x          # fp32 addition, as on the GPU
    assert (xo.cpu().numpy() == xs).all()
    u_ref, bits_ref = oracle_mod.rmsnorm(xs.astype(np.float64), 1e-5)
    check_bf16_rounding(u_ref, bits_ref, u.cpu().numpy())


def test_residual_rmsnorm_in_place_and_add_only(oracle_mod):
    import torch
    rng = np.random.default_rng(9)
    T, d = 4, 512
    x = rng.standard_normal((T, d)).astype(np.float32)
    y = rng.standard_normal((T, d)).astype(np.float32)
    xd, yd = torch.from_numpy(x).cuda(), torch.from_numpy(y).cuda()
    u = torch.zeros((T, d), dtype=torch.int16, device="cuda")
    pp.prunepath_residual_rmsnorm(xd, yd, xd, T, d, 0.0, u)     # x += y in place
    pp.prunepath_residual_rmsnorm(xd, yd, xd, T, d, 0.0, None)  # add only: x += y again
    torch.cuda.synchronize()
    assert (xd.cpu().numpy() == (x + y) + y).all()
    u_ref, bits_ref = oracle_mod.rmsnorm((x + y).astype(np.float64), 0.0)
    check_bf16_rounding(u_ref, bits_ref, u.cpu().numpy())
    with pytest.raises(pp.PrunePathError):
        pp.prunepath_residual_rmsnorm(xd, None, xd, T, 6, 1e-5, u)      # d % 4 != 0
    with pytest.raises(pp.PrunePathError):
        pp.prunepath_residual_rmsnorm(xd, None, xd, T, d, -1.0, u)      # eps < 0


def host_layer(w, l):
    W = make_layer_device(w.d, w.d_ff, w.E, stack_layer_seed(l))
    a = {k: v.cpu().numpy().view(np.uint16) for k, v in W.items()}
    return Layer(w.d, w.d_ff, w.E, a["W_r"], a["W_gate"], a["W_up"], a["W_down"])


def test_stack32_teacher_forced(oracle_mod):
    import torch
    w = WORKLOADS["llama8b_stack32"]
    T, tau = w.T[0], w.taus[0]
    handles = []
    try:
        for l in range(w.layers):
            W = make_layer_device(w.d, w.d_ff, w.E, stack_layer_seed(l))
            handles.append(pp.prunepath_create(w.d, w.d_ff, w.E, T, W["W_r"], W["W_gate"],
                                               W["W_up"], W["W_down"]))
            del W
        S = DecodeStack(handles, w.d, w.E, T, tau)
        x0_bits, _ = workload_tokens(w, T)
        x0 = torch.from_numpy(bf16_to_f32(x0_bits).copy()).cuda()
        S.set_input(x0)
        S.enqueue()
        torch.cuda.synchronize()
        names = ("xs", "us", "ys", "idx", "cnt")
        eager = {k: getattr(S, k).cpu().numpy() for k in names}
        # graph replays, with eager work and synchronisation in between
        S.capture()
        for r in range(3):
            for k in names:
                getattr(S, k).zero_()
            S.set_input(x0)
            S.replay()
            torch.cuda.synchronize()
            for k in names:
                assert (getattr(S, k).cpu().numpy() == eager[k]).all(), (r, k)
            junk = torch.randn(1 << 20, device="cuda").sum().item()
            assert np.isfinite(junk)
    finally:
        for h in handles:
            pp.prunepath_destroy(h)
    xs, us, ys, idx, cnt = (eager[k] for k in names)
    # the residual stream: x_{l+1} = x_l + y_l exactly (fp32), x_0 = input
    assert (xs[0] == bf16_to_f32(x0_bits)).all()
    assert (xs[1:] == xs[:-1] + ys).all()
    # every layer's normalised input against the oracle's RMSNorm of the GPU residual
    ties = 0
    for l in range(w.layers):
        u_ref, bits_ref = oracle_mod.rmsnorm(xs[l].astype(np.float64), 1e-5)
        ties += check_bf16_rounding(u_ref, bits_ref, us[l])
    # sampled layers, teacher-forced: selection and y on the GPU's own input
    ks = []
    for l in (0, 1, 13, 30, 31):
        L = host_layer(w, l)
        u_bits = us[l].view(np.uint16)
        r, _, _ = check_selection(oracle_mod, L, u_bits, tau, 0, idx[l], cnt[l],
                                  label="stack32 layer %d" % l, max_exempt=full_size_cap(w.T[0]))
        check_output(oracle_mod, L, u_bits, 0, idx[l], cnt[l], ys[l], r["g"])
        ks.append(cnt[l].mean())
    union = [len(np.unique(idx[l][idx[l] >= 0])) for l in range(w.layers)]
    print("stack32: mean k per layer %.2f, union %.1f of %d, bf16 ties %d"
          % (cnt.mean(), np.mean(union), w.E, ties))
    assert (cnt >= 1).all() and (cnt <= w.E).all()
