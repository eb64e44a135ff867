"""ctypes binding of libprunepath.so -- argument marshalling only.

Every function has the name and argument order of the C entry point declared
in include/prunepath.h.  Array arguments may be torch tensors on the current
HIP device (their data pointer is passed; bf16 arrays may be typed bfloat16,
int16 or uint16) or raw integer device addresses.  A non-OK status raises
PrunePathError.  There is no fallback: if the shared library is missing the
import fails.
"""
import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libprunepath.so")

PP_OK = 0
PP_EINVAL = 1
PP_ENOMEM = 2
PP_EHIP = 3
PP_EUNSUPPORTED = 4
PP_ENOTCONVERGED = 5

PP_SELECT_NUCLEUS = 0
PP_SELECT_STRICT = 1
PP_SELECT_TOPK = 4
PP_SELECT_LTE = 8
PP_AGG_SUM = 0
PP_AGG_SIGMOID = 2

PP_KERNEL_ROUTE = 0
PP_KERNEL_DISPATCH = 1
PP_KERNEL_GATEUP = 2
PP_KERNEL_DOWN = 3
PP_KERNEL_COUNT = 4

EXPORTED = ("prunepath_create", "prunepath_create_mlp", "prunepath_route", "prunepath_ffn_decode",
            "prunepath_ffn_prefill", "prunepath_destroy", "prunepath_status_string",
            "prunepath_profile_begin", "prunepath_profile_end", "prunepath_residual_rmsnorm",
            "prunepath_router_loss_workspace", "prunepath_router_loss",
            "prunepath_router_loss_noalloc",
            "prunepath_kmeans_workspace", "prunepath_balanced_kmeans")


class PrunePathError(RuntimeError):
    def __init__(self, status, where):
        self.status = status
        super().__init__("%s: %s (status %d)" % (where, _status_text(status), status))


_lib = None


def load():
    """Load the HIP library (raises OSError if it has not been built).

    torch is imported first: its wheel carries its own HIP runtime, which the
    process must share with the library.  Both runtimes have the soname
    libamdhip64.so.7, but torch asks for it by the unversioned name, so a
    library loaded before torch would bind to the system runtime and torch
    would then map its own: device memory from one runtime and kernel launches
    on the other fail."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise OSError("libprunepath.so not built: run __graft_entry__.build() "
                          "or python paper_2605_28283_amd/build.py")
        import torch  # noqa: F401  (maps torch's HIP runtime before the library's dependency)
        lib = ctypes.CDLL(LIB_PATH)
        P, I32, U32, F32 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_uint32, ctypes.c_float
        lib.prunepath_create.argtypes = [ctypes.POINTER(ctypes.c_void_p), I32, I32, I32, I32,
                                         P, P, P, P, P, P, U32, P]
        lib.prunepath_create.restype = ctypes.c_int
        lib.prunepath_create_mlp.argtypes = [ctypes.POINTER(ctypes.c_void_p), I32, I32, I32, I32,
                                             P, P, P, P, P, P, P, U32, P]
        lib.prunepath_create_mlp.restype = ctypes.c_int
        lib.prunepath_route.argtypes = [P, P, I32, F32, P, P, P, P, P]
        lib.prunepath_route.restype = ctypes.c_int
        for f in (lib.prunepath_ffn_decode, lib.prunepath_ffn_prefill):
            f.argtypes = [P, P, I32, F32, P, P, P, P, P]
            f.restype = ctypes.c_int
        lib.prunepath_destroy.argtypes = [P]
        lib.prunepath_destroy.restype = None
        lib.prunepath_profile_begin.argtypes = [P, I32]
        lib.prunepath_profile_begin.restype = ctypes.c_int
        lib.prunepath_profile_end.argtypes = [P, ctypes.POINTER(ctypes.c_double),
                                              ctypes.POINTER(ctypes.c_int32)]
        lib.prunepath_profile_end.restype = ctypes.c_int
        lib.prunepath_residual_rmsnorm.argtypes = [P, P, P, I32, I32, F32, P, P]
        lib.prunepath_residual_rmsnorm.restype = ctypes.c_int
        lib.prunepath_router_loss_workspace.argtypes = [I32, I32]
        lib.prunepath_router_loss_workspace.restype = ctypes.c_size_t
        lib.prunepath_router_loss.argtypes = [P, I32, I32, F32, F32, F32, F32, P, P, P, P]
        lib.prunepath_router_loss.restype = ctypes.c_int
        lib.prunepath_router_loss_noalloc.argtypes = [P, I32, I32, F32, F32, F32, F32, P, P, P]
        lib.prunepath_router_loss_noalloc.restype = ctypes.c_int
        lib.prunepath_kmeans_workspace.argtypes = [I32, I32, I32]
        lib.prunepath_kmeans_workspace.restype = ctypes.c_size_t
        lib.prunepath_balanced_kmeans.argtypes = [P, I32, I32, I32, P, I32, P, P, P, P, P, P, P,
                                                  P]
        lib.prunepath_balanced_kmeans.restype = ctypes.c_int
        lib.prunepath_status_string.argtypes = [ctypes.c_int]
        lib.prunepath_status_string.restype = ctypes.c_char_p
        _lib = lib
    return _lib


def _status_text(s):
    try:
        return load().prunepath_status_string(int(s)).decode()
    except OSError:
        return "unknown"


_BF16_LIKE = None


def _ptr(a, kind=None):
    """Device address of a tensor (checked) or an int; None -> NULL."""
    if a is None:
        return None
    if isinstance(a, int):
        return a
    import torch
    global _BF16_LIKE
    if _BF16_LIKE is None:
        _BF16_LIKE = {torch.bfloat16, torch.int16, torch.uint16}
    if not a.is_cuda:
        raise ValueError("array arguments must live on the GPU")
    if not a.is_contiguous():
        raise ValueError("array arguments must be contiguous")
    want = {"bf16": _BF16_LIKE, "f32": {torch.float32}, "i32": {torch.int32}}.get(kind)
    if want is not None and a.dtype not in want:
        raise TypeError("expected %s array, got %s" % (kind, a.dtype))
    return a.data_ptr()


def _stream(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _check(st, where):
    if st != PP_OK:
        raise PrunePathError(st, where)


def prunepath_status_string(status):
    return _status_text(status)


def prunepath_create(d, d_ff, E, max_tokens, W_r, W_gate, W_up, W_down, perm=None,
                     router_bias=None, flags=0, stream=None):
    """Returns an opaque handle (int)."""
    out = ctypes.c_void_p()
    st = load().prunepath_create(ctypes.byref(out), d, d_ff, E, max_tokens,
                                 _ptr(W_r, "bf16"), _ptr(W_gate, "bf16"), _ptr(W_up, "bf16"),
                                 _ptr(W_down, "bf16"), _ptr(perm, "i32"),
                                 _ptr(router_bias, "f32"), flags, _stream(stream))
    _check(st, "prunepath_create")
    return out.value


def prunepath_create_mlp(d, d_ff, E, max_tokens, W_r, W_fc, b_fc, W_proj, b_proj, perm=None,
                         router_bias=None, flags=0, stream=None):
    """Non-gated GELU MLP layer (b_fc / b_proj may be None).  Returns a handle."""
    out = ctypes.c_void_p()
    st = load().prunepath_create_mlp(ctypes.byref(out), d, d_ff, E, max_tokens,
                                     _ptr(W_r, "bf16"), _ptr(W_fc, "bf16"), _ptr(b_fc, "f32"),
                                     _ptr(W_proj, "bf16"), _ptr(b_proj, "f32"), _ptr(perm, "i32"),
                                     _ptr(router_bias, "f32"), flags, _stream(stream))
    _check(st, "prunepath_create_mlp")
    return out.value


def prunepath_route(handle, x, T, tau, inv_temp, expert_idx, count, gate_w=None, stream=None):
    st = load().prunepath_route(handle, _ptr(x, "bf16"), T, tau, _ptr(inv_temp, "f32"),
                                _ptr(expert_idx, "i32"), _ptr(count, "i32"),
                                _ptr(gate_w, "f32"), _stream(stream))
    _check(st, "prunepath_route")


def prunepath_ffn_decode(handle, x, T, tau, inv_temp, y, expert_idx=None, count=None,
                         stream=None):
    st = load().prunepath_ffn_decode(handle, _ptr(x, "bf16"), T, tau, _ptr(inv_temp, "f32"),
                                     _ptr(y, "f32"), _ptr(expert_idx, "i32"), _ptr(count, "i32"),
                                     _stream(stream))
    _check(st, "prunepath_ffn_decode")


def prunepath_ffn_prefill(handle, x, T, tau, inv_temp, y, expert_idx=None, count=None,
                          stream=None):
    st = load().prunepath_ffn_prefill(handle, _ptr(x, "bf16"), T, tau, _ptr(inv_temp, "f32"),
                                      _ptr(y, "f32"), _ptr(expert_idx, "i32"),
                                      _ptr(count, "i32"), _stream(stream))
    _check(st, "prunepath_ffn_prefill")


def prunepath_residual_rmsnorm(x, y, x_out, T, d, eps, u=None, stream=None):
    st = load().prunepath_residual_rmsnorm(_ptr(x, "f32"), _ptr(y, "f32"), _ptr(x_out, "f32"),
                                           T, d, eps, _ptr(u, "bf16"), _stream(stream))
    _check(st, "prunepath_residual_rmsnorm")


def prunepath_router_loss_workspace(B, E):
    """Workspace bytes prunepath_router_loss needs (0 for bad sizes)."""
    return int(load().prunepath_router_loss_workspace(B, E))


def prunepath_router_loss(g, B, E, eps, eta, lam, gamma, losses, dg, workspace, stream=None):
    """losses[4] = [L_ent, L_bal, L_gate, total] and dg = dL/dg (None: skipped)."""
    st = load().prunepath_router_loss(_ptr(g, "f32"), B, E, eps, eta, lam, gamma,
                                      _ptr(losses, "f32"), _ptr(dg, "f32"), _ptr(workspace),
                                      _stream(stream))
    _check(st, "prunepath_router_loss")


def prunepath_router_loss_noalloc(g, B, E, eps, eta, lam, gamma, losses, dg, stream=None):
    """prunepath_router_loss with the library's own device scratch (no
    workspace argument, nothing allocated)."""
    st = load().prunepath_router_loss_noalloc(_ptr(g, "f32"), B, E, eps, eta, lam, gamma,
                                              _ptr(losses, "f32"), _ptr(dg, "f32"),
                                              _stream(stream))
    _check(st, "prunepath_router_loss_noalloc")


def prunepath_kmeans_workspace(n, D, k):
    """Workspace bytes prunepath_balanced_kmeans needs (0 for bad sizes)."""
    return int(load().prunepath_kmeans_workspace(n, D, k))


def prunepath_balanced_kmeans(F, n, D, k, init_centroids, iters, assign, perm, centroids,
                              workspace, objective=None, prices=None, stream=None):
    """Balanced k-means of F's rows (blocks until done).  Returns the auction
    rounds of each iteration as a list."""
    rounds = (ctypes.c_int32 * iters)()
    st = load().prunepath_balanced_kmeans(
        _ptr(F, "bf16"), n, D, k, _ptr(init_centroids, "f32"), iters, _ptr(assign, "i32"),
        _ptr(perm, "i32"), _ptr(centroids, "f32"), _ptr(objective, "f32"), _ptr(prices, "f32"),
        ctypes.cast(rounds, ctypes.c_void_p), _ptr(workspace), _stream(stream))
    _check(st, "prunepath_balanced_kmeans")
    return list(rounds)


def prunepath_profile_begin(handle, capacity):
    _check(load().prunepath_profile_begin(handle, capacity), "prunepath_profile_begin")


def prunepath_profile_end(handle):
    """Returns (ms[PP_KERNEL_COUNT], launches[PP_KERNEL_COUNT]) as lists."""
    ms = (ctypes.c_double * PP_KERNEL_COUNT)()
    n = (ctypes.c_int32 * PP_KERNEL_COUNT)()
    _check(load().prunepath_profile_end(handle, ms, n), "prunepath_profile_end")
    return list(ms), list(n)


def prunepath_destroy(handle):
    if handle:
        load().prunepath_destroy(handle)
