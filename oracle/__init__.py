"""PrunePath sparse-FFN forward: CPU oracle (fp64) -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The HIP library never calls it and it
never calls the HIP library; the two share only the seeded bf16 inputs.

The arithmetic lives in ``prunepath_oracle.c`` (fp64, per token, following the
paper's Sec. 3.1 equations in order, and the Sec. 3.2 / Sec. 4.2.3 routing
regularisers with their gradient); this module only marshals numpy arrays.

The balanced k-means of MoEfication's clustering step (Sec. 2.2) is the
module ``oracle.kmeans`` (numpy / scipy, fp64).

Readings taken where the paper is open are stated in the C file's header.
Every function here is pinned by ``tests/test_oracle_pins.py`` against closed
forms, library routines, brute force and the paper's all-expert identity
(Eq. moefication_decomp).
"""
import ctypes
import os

import numpy as np

from . import build as _build

SELECT_NUCLEUS = 0
SELECT_STRICT = 1
SELECT_TOPK = 4
SELECT_LTE = 8
AGG_SUM = 0
AGG_SIGMOID = 2

_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_build.LIB) or (
                os.path.getmtime(_build.LIB) < os.path.getmtime(_build.SRC)):
            _build.build()
        lib = ctypes.CDLL(_build.LIB)
        P = ctypes.c_void_p
        I64 = ctypes.c_int64
        lib.ppo_route.argtypes = [I64, I64, I64, P, P, P, P, ctypes.c_double, ctypes.c_uint,
                                  P, P, P, P]
        lib.ppo_route.restype = ctypes.c_int
        lib.ppo_ffn.argtypes = [I64, I64, I64, I64, P, P, P, P, P, P, P, P, ctypes.c_uint, P]
        lib.ppo_ffn.restype = ctypes.c_int
        lib.ppo_softmax.argtypes = [I64, P, P]
        lib.ppo_softmax.restype = None
        lib.ppo_order.argtypes = [I64, P, P]
        lib.ppo_order.restype = None
        lib.ppo_cut.argtypes = [I64, P, ctypes.c_double, ctypes.c_uint, P]
        lib.ppo_cut.restype = I64
        lib.ppo_bf16_round_n.argtypes = [I64, P, P]
        lib.ppo_bf16_round_n.restype = None
        lib.ppo_rmsnorm.argtypes = [I64, I64, P, ctypes.c_double, P, P]
        lib.ppo_rmsnorm.restype = ctypes.c_int
        lib.ppo_mlp.argtypes = [I64, I64, I64, I64, P, P, P, P, P, P, P, P, P, ctypes.c_uint, P]
        lib.ppo_mlp.restype = ctypes.c_int
        lib.ppo_gelu_n.argtypes = [I64, P, P]
        lib.ppo_gelu_n.restype = None
        lib.ppo_router_loss.argtypes = [I64, I64, P, ctypes.c_double, ctypes.c_double,
                                        ctypes.c_double, ctypes.c_double, P, P]
        lib.ppo_router_loss.restype = ctypes.c_int
        lib.ppo_num_threads.argtypes = []
        lib.ppo_num_threads.restype = ctypes.c_int
        lib.ppo_set_num_threads.argtypes = [ctypes.c_int]
        lib.ppo_set_num_threads.restype = None
        _lib = lib
    return _lib


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dtype):
    return None if a is None else np.ascontiguousarray(a, dtype=dtype)


def num_threads() -> int:
    return _load().ppo_num_threads()


def set_num_threads(n: int) -> None:
    """Threads the oracle's OpenMP loops use from now on (benchmark timing)."""
    _load().ppo_set_num_threads(int(n))


def softmax(g):
    g = _c(g, np.float64)
    p = np.empty_like(g)
    _load().ppo_softmax(g.size, _ptr(g), _ptr(p))
    return p


def order(g):
    g = _c(g, np.float64)
    pi = np.empty(g.size, np.int32)
    _load().ppo_order(g.size, _ptr(g), _ptr(pi))
    return pi


def cut(p_sorted, tau, flags=0):
    """Returns (k, C) for probabilities already in descending order."""
    p = _c(p_sorted, np.float64)
    C = np.empty_like(p)
    k = _load().ppo_cut(p.size, _ptr(p), float(tau), int(flags), _ptr(C))
    return int(k), C


def route(x, W_r, tau, flags=0, bias=None, inv_temp=None):
    """Routing of T tokens.  x: [T,d] uint16 (bf16 bits), W_r: [E,d] uint16.

    Returns dict(idx [T,E] int32 (-1 padded), count [T] int32, g [T,E] fp64
    logits, cum [T,E] fp64 cumulative mass in selection order)."""
    x = _c(x, np.uint16)
    W_r = _c(W_r, np.uint16)
    T, d = x.shape
    E = W_r.shape[0]
    assert W_r.shape[1] == d
    bias = _c(bias, np.float32)
    inv_temp = _c(inv_temp, np.float32)
    idx = np.empty((T, E), np.int32)
    count = np.empty(T, np.int32)
    g = np.empty((T, E), np.float64)
    cum = np.empty((T, E), np.float64)
    rc = _load().ppo_route(T, d, E, _ptr(x), _ptr(W_r), _ptr(bias), _ptr(inv_temp), float(tau),
                           int(flags), _ptr(idx), _ptr(count), _ptr(g), _ptr(cum))
    if rc != 0:
        raise ValueError("oracle route: bad arguments")
    return dict(idx=idx, count=count, g=g, cum=cum)


def ffn(x, W_gate, W_up, W_down, idx, count, flags=0, g=None, perm=None):
    """y [T,d] fp64 for a given selection (idx [T,E] -1 padded, count [T])."""
    x = _c(x, np.uint16)
    T, d = x.shape
    d_ff = W_gate.shape[0]
    E = idx.shape[1]
    assert W_gate.shape == (d_ff, d) and W_up.shape == (d_ff, d) and W_down.shape == (d, d_ff)
    y = np.empty((T, d), np.float64)
    rc = _load().ppo_ffn(T, d, d_ff, E, _ptr(x), _ptr(_c(W_gate, np.uint16)),
                         _ptr(_c(W_up, np.uint16)), _ptr(_c(W_down, np.uint16)),
                         _ptr(_c(perm, np.int32)), _ptr(_c(idx, np.int32)),
                         _ptr(_c(count, np.int32)), _ptr(_c(g, np.float64)), int(flags), _ptr(y))
    if rc != 0:
        raise ValueError("oracle ffn: bad arguments")
    return y


def gelu(a):
    """GPT-2's tanh-form GELU, elementwise, fp64."""
    a = _c(a, np.float64)
    out = np.empty_like(a)
    _load().ppo_gelu_n(a.size, _ptr(a), _ptr(out))
    return out


def mlp(x, W_fc, b_fc, W_proj, b_proj, idx, count, flags=0, g=None, perm=None):
    """Non-gated GELU MLP variant: y [T,d] fp64 for a given selection; b_fc
    [d_ff] / b_proj [d] fp32 or None."""
    x = _c(x, np.uint16)
    T, d = x.shape
    d_ff = W_fc.shape[0]
    E = idx.shape[1]
    assert W_fc.shape == (d_ff, d) and W_proj.shape == (d, d_ff)
    y = np.empty((T, d), np.float64)
    rc = _load().ppo_mlp(T, d, d_ff, E, _ptr(x), _ptr(_c(W_fc, np.uint16)),
                         _ptr(_c(b_fc, np.float32)), _ptr(_c(W_proj, np.uint16)),
                         _ptr(_c(b_proj, np.float32)), _ptr(_c(perm, np.int32)),
                         _ptr(_c(idx, np.int32)), _ptr(_c(count, np.int32)),
                         _ptr(_c(g, np.float64)), int(flags), _ptr(y))
    if rc != 0:
        raise ValueError("oracle mlp: bad arguments")
    return y


def forward(x, W_r, W_gate, W_up, W_down, tau, flags=0, bias=None, inv_temp=None, perm=None):
    """Routing followed by the selected experts' outputs; returns (route dict, y)."""
    r = route(x, W_r, tau, flags=flags, bias=bias, inv_temp=inv_temp)
    y = ffn(x, W_gate, W_up, W_down, r["idx"], r["count"], flags=flags, g=r["g"], perm=perm)
    return r, y


def near_tie(cum, tau, band=1e-5, flags=0):
    """Cumulative-mass ties of the cut (Eq. tau_thresh_activate): tokens whose
    cumulative mass lies within `band` of tau at some cut position
    (C_1..C_{E-1}; C_E = 1 decides nothing for tau < 1).  For these the count
    may legitimately differ between fp32 and fp64 evaluation.  Nothing is near
    a tie when the rule keeps every expert regardless of C (nucleus with
    tau >= 1, strict with tau > 1), nor for the top-k and LTE rules, which do
    not read C."""
    cum = np.asarray(cum)
    if flags & (SELECT_TOPK | SELECT_LTE):
        return np.zeros(cum.shape[0], bool)
    if (flags & SELECT_STRICT and tau > 1.0) or (not flags & SELECT_STRICT and tau >= 1.0):
        return np.zeros(cum.shape[0], bool)
    return (np.abs(cum[:, :-1] - tau) <= band).any(axis=1)


def lte_tie(g, delta, band=1e-6):
    """LTE threshold ties (Eq. lte_hard_set): tokens with an expert whose
    sigmoid score lies within `band` of delta; their kept set may differ
    between fp32 and fp64 evaluation."""
    s = 1.0 / (1.0 + np.exp(-np.asarray(g, np.float64)))
    return (np.abs(s - delta) <= band).any(axis=1)


def _sorted_desc(g):
    g = np.asarray(g, np.float64)
    return -np.sort(-g, axis=1)


def cut_order_tie(g, count, band=1e-5):
    """Logit ties at the cut: tokens whose last kept and first dropped experts
    in the descending order (pi_k, pi_{k+1}) have logits within `band`.
    Which of the two is kept is then not unique under fp32 evaluation (the
    count is not affected unless the mass is also near tau).  Tokens keeping
    no expert or all E have no cut."""
    srt = _sorted_desc(g)
    T, E = srt.shape
    k = np.asarray(count, np.int64)
    out = np.zeros(T, bool)
    rows = np.nonzero((k >= 1) & (k < E))[0]
    out[rows] = srt[rows, k[rows] - 1] - srt[rows, k[rows]] <= band
    return out


def prefix_order_tie(g, count, band=1e-5):
    """Logit ties inside the kept prefix: tokens with two consecutive kept
    experts whose logits lie within `band`.  The kept set stays unique (a
    swap inside the prefix changes C only at positions within `band` of
    tau, which near_tie covers), but the order in which the kept experts are
    listed is not."""
    srt = _sorted_desc(g)
    T, E = srt.shape
    k = np.asarray(count, np.int64)
    out = np.zeros(T, bool)
    for t in range(T):
        if k[t] >= 2:
            out[t] = bool((srt[t, :k[t] - 1] - srt[t, 1:k[t]] <= band).any())
    return out


def bf16_round(v):
    """bf16 bit patterns nearest to fp64 values (ties to even, one rounding)."""
    v = _c(v, np.float64)
    out = np.empty(v.shape, np.uint16)
    _load().ppo_bf16_round_n(v.size, _ptr(v), _ptr(out))
    return out


def rmsnorm(x, eps=1e-5):
    """Pre-norm of the stacked workload: returns (u fp64 [T,d], u bf16 bits)."""
    x = _c(x, np.float64)
    T, d = x.shape
    u = np.empty_like(x)
    bits = np.empty(x.shape, np.uint16)
    if _load().ppo_rmsnorm(T, d, _ptr(x), float(eps), _ptr(u), _ptr(bits)) != 0:
        raise ValueError("oracle rmsnorm: bad arguments")
    return u, bits


def router_loss(g, eps=1e-8, eta=1.0, lam=1.0, gamma=0.0, grad=True):
    """Routing regularisers over a batch of router logits g [B, E] (Sec. 3.2
    and Sec. 4.2.3): returns (losses, dg) with losses = [L_ent, L_bal, L_gate,
    eta L_ent + lam L_bal + gamma L_gate] and dg = dL/dg [B, E] (None when
    grad is False)."""
    g = _c(g, np.float64)
    B, E = g.shape
    losses = np.empty(4)
    dg = np.empty_like(g) if grad else None
    if _load().ppo_router_loss(B, E, _ptr(g), float(eps), float(eta), float(lam), float(gamma),
                               _ptr(losses), _ptr(dg)) != 0:
        raise ValueError("oracle router_loss: bad arguments")
    return losses, dg
