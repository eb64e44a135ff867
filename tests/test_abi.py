"""CPU-side checks of the C ABI: the library loads, exports every entry point
declared in include/prunepath.h, and rejects bad arguments on the host before
touching the GPU (these calls return before any HIP runtime call)."""
import ctypes
import os
import re

import pytest

import paper_2605_28283_amd as pp

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "prunepath.h")


def declared_symbols():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(prunepath_\w+)\s*\(", text)))


def test_header_declares_the_five_calls():
    syms = declared_symbols()
    for s in ("prunepath_create", "prunepath_route", "prunepath_ffn_decode",
              "prunepath_ffn_prefill", "prunepath_destroy"):
        assert s in syms


def test_library_exports_every_declared_symbol():
    lib = pp.load()
    for s in declared_symbols():
        assert hasattr(lib, s), s
    # and the binding exposes the same names
    for s in declared_symbols():
        assert callable(getattr(pp, s)), s
    assert sorted(pp.EXPORTED) == declared_symbols()


def test_status_strings():
    for code, text in ((pp.PP_OK, "ok"), (pp.PP_EINVAL, "invalid argument"),
                       (pp.PP_EUNSUPPORTED, "unsupported shape")):
        assert pp.prunepath_status_string(code) == text
    assert pp.prunepath_status_string(99) == "unknown status"


def _create(**kw):
    lib = pp.load()
    a = dict(d=512, d_ff=2048, E=16, max_tokens=8, W_r=8, W_gate=8, W_up=8, W_down=8, perm=None,
             bias=None, flags=0)
    a.update(kw)
    out = ctypes.c_void_p(1234)
    st = lib.prunepath_create(ctypes.byref(out), a["d"], a["d_ff"], a["E"], a["max_tokens"],
                              a["W_r"], a["W_gate"], a["W_up"], a["W_down"], a["perm"], a["bias"],
                              a["flags"], None)
    return st, out.value


@pytest.mark.parametrize("kw,expect", [
    (dict(W_r=None), pp.PP_EINVAL),
    (dict(W_down=None), pp.PP_EINVAL),
    (dict(d=0), pp.PP_EINVAL),
    (dict(max_tokens=0), pp.PP_EINVAL),
    (dict(max_tokens=70000), pp.PP_EINVAL),
    (dict(flags=16), pp.PP_EINVAL),               # unknown flag bit
    (dict(flags=pp.PP_SELECT_STRICT | pp.PP_SELECT_TOPK), pp.PP_EINVAL),   # two rules
    (dict(flags=pp.PP_SELECT_TOPK | pp.PP_SELECT_LTE | pp.PP_AGG_SIGMOID), pp.PP_EINVAL),
    (dict(d_ff=2050), pp.PP_EINVAL),
    (dict(d_ff=4096), pp.PP_EUNSUPPORTED),        # experts of 256 neurons
    (dict(E=512, d_ff=512 * 128), pp.PP_EUNSUPPORTED),
    (dict(d=520), pp.PP_EUNSUPPORTED),            # d not a multiple of 64
])
def test_create_rejects_bad_arguments(kw, expect):
    st, h = _create(**kw)
    assert st == expect
    assert h is None or h == 0


def test_create_null_out():
    lib = pp.load()
    assert lib.prunepath_create(None, 512, 2048, 16, 8, 8, 8, 8, 8, None, None, 0, None) == \
        pp.PP_EINVAL


def test_calls_reject_null_handle():
    lib = pp.load()
    assert lib.prunepath_route(None, 8, 1, 0.5, None, 8, 8, None, None) == pp.PP_EINVAL
    assert lib.prunepath_ffn_decode(None, 8, 1, 0.5, None, 8, None, None, None) == pp.PP_EINVAL
    assert lib.prunepath_ffn_prefill(None, 8, 1, 0.5, None, 8, None, None, None) == pp.PP_EINVAL
    lib.prunepath_destroy(None)  # NULL-safe


def test_binding_raises_on_error():
    with pytest.raises(pp.PrunePathError) as ei:
        pp.prunepath_route(0, 8, 1, 0.5, None, 8, 8, stream=0)
    assert ei.value.status == pp.PP_EINVAL


@pytest.mark.parametrize("args", [
    (None, None, 16, 4, 64, 1e-5, 8),          # x NULL
    (16, None, None, 4, 64, 1e-5, 8),          # x_out NULL
    (16, None, 16, 0, 64, 1e-5, 8),            # T < 1
    (16, None, 16, 4, 66, 1e-5, 8),            # d % 4 != 0
    (16, None, 16, 4, 0, 1e-5, 8),             # d < 4
    (16, None, 16, 4, 64, float("nan"), 8),    # eps NaN
    (16, None, 16, 4, 64, -1.0, 8),            # eps < 0
    (8, None, 24, 4, 64, 1e-5, 8),             # x_out not 16-byte aligned
    (16, None, 16, 4, 64, 1e-5, 4),            # u not 8-byte aligned
])
def test_residual_rmsnorm_rejects_bad_arguments(args):
    lib = pp.load()
    x, y, xo, T, d, eps, u = args
    assert lib.prunepath_residual_rmsnorm(x, y, xo, T, d, eps, u, None) == pp.PP_EINVAL


def test_router_loss_workspace_size():
    lib = pp.load()
    for B, E in [(1, 1), (16, 112), (17, 112), (16384, 256), (1 << 22, 256)]:
        nb = -(-B // 64)
        assert lib.prunepath_router_loss_workspace(B, E) == 4 * nb * (E + 2)
    for B, E in [(0, 8), (8, 0), (8, 257), ((1 << 22) + 1, 8), (-1, 8)]:
        assert lib.prunepath_router_loss_workspace(B, E) == 0


INF, NAN = float("inf"), float("nan")


@pytest.mark.parametrize("args", [
    (None, 8, 16, 1e-8, 1.0, 1.0, 0.0, 16, 32, 64),     # g NULL
    (16, 8, 16, 1e-8, 1.0, 1.0, 0.0, None, 32, 64),     # losses NULL
    (16, 8, 16, 1e-8, 1.0, 1.0, 0.0, 16, 32, None),     # workspace NULL
    (16, 8, 16, 1e-8, 1.0, 1.0, 0.0, 48, 16, 64),       # dg aliases g
    (16, 0, 16, 1e-8, 1.0, 1.0, 0.0, 48, 32, 64),       # B < 1
    (16, (1 << 22) + 1, 16, 1e-8, 1.0, 1.0, 0.0, 48, 32, 64),  # B too large
    (16, 8, 0, 1e-8, 1.0, 1.0, 0.0, 48, 32, 64),        # E < 1
    (16, 8, 257, 1e-8, 1.0, 1.0, 0.0, 48, 32, 64),      # E > 256
    (16, 8, 16, -1e-8, 1.0, 1.0, 0.0, 48, 32, 64),      # eps < 0
    (16, 8, 16, NAN, 1.0, 1.0, 0.0, 48, 32, 64),        # eps NaN
    (16, 8, 16, INF, 1.0, 1.0, 0.0, 48, 32, 64),        # eps infinite
    (16, 8, 16, 1e-8, NAN, 1.0, 0.0, 48, 32, 64),       # eta NaN
    (16, 8, 16, 1e-8, 1.0, INF, 0.0, 48, 32, 64),       # lambda infinite
    (16, 8, 16, 1e-8, 1.0, 1.0, -INF, 48, 32, 64),      # gamma infinite
    (18, 8, 16, 1e-8, 1.0, 1.0, 0.0, 48, 32, 64),       # g misaligned
    (16, 8, 16, 1e-8, 1.0, 1.0, 0.0, 48, 32, 66),       # workspace misaligned
    (16, 8, 16, 1e-8, 1.0, 1.0, 0.0, 48, 40, 64),       # dg not 16-byte aligned
    (24, 8, 16, 1e-8, 1.0, 1.0, 0.0, 48, 32, 64),       # g not 16-byte aligned
])
def test_router_loss_rejects_bad_arguments(args):
    lib = pp.load()
    g, B, E, eps, eta, lam, gam, losses, dg, ws = args
    assert lib.prunepath_router_loss(g, B, E, eps, eta, lam, gam, losses, dg, ws,
                                     None) == pp.PP_EINVAL


@pytest.mark.parametrize("args", [
    (None, 8, 8),      # W_r NULL
    (8, None, 8),      # W_fc NULL
    (8, 8, None),      # W_proj NULL
])
def test_create_mlp_rejects_null_weights(args):
    import ctypes
    lib = pp.load()
    W_r, W_fc, W_proj = args
    out = ctypes.c_void_p(123)
    assert lib.prunepath_create_mlp(ctypes.byref(out), 64, 128, 1, 4, W_r, W_fc, None, W_proj,
                                    None, None, None, 0, None) == pp.PP_EINVAL
    assert out.value is None


def test_create_mlp_rejects_bad_shapes():
    import ctypes
    lib = pp.load()
    out = ctypes.c_void_p()
    for d, d_ff, E, mt, flags, want in ((0, 128, 1, 4, 0, pp.PP_EINVAL),
                                        (64, 128, 1, 0, 0, pp.PP_EINVAL),
                                        (64, 256, 1, 4, 0, pp.PP_EUNSUPPORTED),
                                        (96, 128, 1, 4, 0, pp.PP_EUNSUPPORTED),
                                        (64, 128, 1, 4, 16, pp.PP_EINVAL)):
        assert lib.prunepath_create_mlp(ctypes.byref(out), d, d_ff, E, mt, 8, 8, None, 8, None,
                                        None, None, flags, None) == want


def test_kmeans_workspace_and_rejections():
    lib = pp.load()
    assert lib.prunepath_kmeans_workspace(14336, 4096, 112) > 0
    for n, D, k in ((0, 64, 1), (64, 64, 0), (64, 64, 257), (100, 64, 8), (64, 96, 8),
                    (64, 32, 8), (131072, 64, 8), (8, 64, 16)):
        assert lib.prunepath_kmeans_workspace(n, D, k) == 0, (n, D, k)
    args = dict(F=16, n=256, D=64, k=8, init=16, iters=1, assign=16, perm=16, cent=16, ws=256)
    bad = [dict(F=None), dict(init=None), dict(assign=None), dict(perm=None), dict(cent=None),
           dict(ws=None), dict(iters=0), dict(iters=1001), dict(n=100), dict(D=96), dict(k=0),
           dict(F=8), dict(ws=264)]
    for b in bad:
        a = dict(args, **b)
        st = lib.prunepath_balanced_kmeans(a["F"], a["n"], a["D"], a["k"], a["init"], a["iters"],
                                           a["assign"], a["perm"], a["cent"], None, None, None,
                                           a["ws"], None)
        assert st == pp.PP_EINVAL, b
    assert pp.prunepath_status_string(pp.PP_ENOTCONVERGED) == "did not converge"


def test_one_hip_runtime_whatever_the_import_order():
    """Loading the library before torch must not map a second HIP runtime
    (torch's wheel carries its own; both would serve the same GPU with
    separate state, and launches on pointers from the other one fail)."""
    import subprocess
    import sys
    code = ("import paper_2605_28283_amd as pp; pp.load(); import torch; "
            "print(len(set(l.split()[-1] for l in open('/proc/self/maps') "
            "if 'libamdhip64' in l)))")
    r = subprocess.run([sys.executable, "-c", code], cwd=ROOT, capture_output=True, text=True,
                       timeout=300)
    assert r.returncode == 0, r.stderr
    assert r.stdout.strip().splitlines()[-1] == "1"
