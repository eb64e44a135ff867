"""Helpers shared by the GPU parity tests: upload seeded layers, run the HIP
entry points through the binding, and compare against the oracle."""
import numpy as np

import paper_2605_28283_amd as pp

TOL = 1e-2          # max |y - y_ref| <= TOL * RMS(y_ref)  (global RMS of the call)
TIE_BAND = 1e-5     # cumulative-mass / logit band treated as a tie
LTE_BAND = 1e-6     # sigmoid-score band around delta treated as a tie (LTE rule)


def torch():
    import torch as _t
    return _t


def to_dev(bits):
    t = torch()
    return t.from_numpy(np.ascontiguousarray(bits).view(np.int16)).cuda()


class DevLayer:
    """A SwiGLU layer (workloads.Layer) or a non-gated GELU MLP layer
    (workloads.MlpLayer) uploaded and created through the C ABI."""

    def __init__(self, L, max_tokens, flags=0, biases=True):
        t = torch()
        self.L = L
        self.flags = flags
        self.E, self.d = L.E, L.d
        self.mlp = hasattr(L, "W_fc")
        self.perm = None if L.perm is None else t.from_numpy(L.perm).cuda()
        self.bias = None if L.bias is None else t.from_numpy(L.bias).cuda()
        if self.mlp:
            self.W = [to_dev(a) for a in (L.W_r, L.W_fc, L.W_proj)]
            self.b_fc = t.from_numpy(L.b_fc).cuda() if biases else None
            self.b_proj = t.from_numpy(L.b_proj).cuda() if biases else None
            self.h = pp.prunepath_create_mlp(L.d, L.d_ff, L.E, max_tokens, self.W[0], self.W[1],
                                             self.b_fc, self.W[2], self.b_proj, perm=self.perm,
                                             router_bias=self.bias, flags=flags)
        else:
            self.W = [to_dev(a) for a in (L.W_r, L.W_gate, L.W_up, L.W_down)]
            self.h = pp.prunepath_create(L.d, L.d_ff, L.E, max_tokens, *self.W, perm=self.perm,
                                         router_bias=self.bias, flags=flags)
        self.biases = biases

    def close(self):
        if self.h:
            pp.prunepath_destroy(self.h)
            self.h = None

    def __enter__(self):
        return self

    def __exit__(self, *a):
        self.close()

    def run(self, mode, x_bits, tau, inv_temp=None):
        """mode: 'decode' | 'prefill' | 'route'.  Returns numpy (idx, count, y or gate_w)."""
        t = torch()
        T = x_bits.shape[0]
        x = to_dev(x_bits)
        it = None if inv_temp is None else t.from_numpy(inv_temp).cuda()
        idx = t.full((T, self.E), -7, dtype=t.int32, device="cuda")
        cnt = t.full((T,), -7, dtype=t.int32, device="cuda")
        if mode == "route":
            gw = t.full((T, self.E), -7.0, dtype=t.float32, device="cuda")
            pp.prunepath_route(self.h, x, T, tau, it, idx, cnt, gw)
            t.cuda.synchronize()
            return idx.cpu().numpy(), cnt.cpu().numpy(), gw.cpu().numpy()
        y = t.full((T, self.d), float("nan"), dtype=t.float32, device="cuda")
        fn = pp.prunepath_ffn_decode if mode == "decode" else pp.prunepath_ffn_prefill
        fn(self.h, x, T, tau, it, y, idx, cnt)
        t.cuda.synchronize()
        return idx.cpu().numpy(), cnt.cpu().numpy(), y.cpu().numpy()


def cut_count(C, tau, strict):
    E = len(C)
    if strict:
        m = int(np.sum(C[:-1] < tau)) + (1 if tau > 1.0 else 0)
        return max(1, m)
    if tau >= 1.0:
        return E
    hit = np.nonzero(C >= tau)[0]
    return int(hit[0]) + 1 if len(hit) else E


def check_tie_token(g, C, tau, flags, kept, oracle):
    """A token inside the tie band: its count must be one that the cut gives
    for some cumulative masses within TIE_BAND of the oracle's, and the kept
    experts must be a prefix of the logit order up to TIE_BAND."""
    strict = bool(flags & oracle.SELECT_STRICT)
    k = len(kept)
    k_lo = cut_count(C + TIE_BAND, tau, strict)
    k_hi = cut_count(C - TIE_BAND, tau, strict)
    assert k_lo <= k <= k_hi, (k, k_lo, k_hi)
    rest = np.setdiff1d(np.arange(len(g)), kept)
    if len(rest):
        assert g[kept].min() >= g[rest].max() - TIE_BAND
    assert (np.diff(g[kept]) <= TIE_BAND).all()


def check_rule_tie_token(g, tau, flags, kept, oracle):
    """Top-k / LTE token inside a tie band: the kept set is a prefix of the
    logit order up to TIE_BAND, of the right size (top-k) or with every kept
    score above and every dropped score below delta up to LTE_BAND (LTE)."""
    E = len(g)
    rest = np.setdiff1d(np.arange(E), kept)
    if len(kept) and len(rest):
        assert g[kept].min() >= g[rest].max() - TIE_BAND
    if flags & oracle.SELECT_TOPK:
        assert len(kept) == min(E, max(1, int(np.floor(tau + 0.5))))
    else:
        s = 1.0 / (1.0 + np.exp(-g))
        assert (s[kept] >= tau - LTE_BAND).all() and (s[rest] <= tau + LTE_BAND).all()


# Per-call tie statistics of the GPU parity checks, printed in the pytest
# terminal summary (tests/conftest.py): (label, T, tau, counts by kind).
TIE_LOG = []

# Largest share of tokens a full-size workload call may exempt from bit-exact
# selection parity (the tie bands make this ~1e-3 on the seeded workloads).
FULL_SIZE_EXEMPT_FRACTION = 0.01


def tie_kinds(oracle, r, tau, flags):
    """Tokens exempt from bit-exact selection, by kind, from the oracle's
    fp64 routing r: 'mass' (cumulative mass within TIE_BAND of tau),
    'cut_order' (last kept and first dropped logits within TIE_BAND; not for
    LTE, whose set is a per-expert threshold), 'lte' (a sigmoid score within
    LTE_BAND of delta).  'prefix_order' (two kept logits within TIE_BAND)
    exempts nothing: the set is still compared exactly, only the listed order
    may differ between tied experts."""
    sel = flags & (oracle.SELECT_STRICT | oracle.SELECT_TOPK | oracle.SELECT_LTE)
    T = r["g"].shape[0]
    k = {"mass": oracle.near_tie(r["cum"], tau, TIE_BAND, flags=sel)}
    if sel & oracle.SELECT_LTE:
        k["cut_order"] = np.zeros(T, bool)
        k["lte"] = oracle.lte_tie(r["g"], tau, LTE_BAND)
    else:
        k["cut_order"] = oracle.cut_order_tie(r["g"], r["count"], TIE_BAND)
        k["lte"] = np.zeros(T, bool)
    k["prefix_order"] = oracle.prefix_order_tie(r["g"], r["count"], TIE_BAND)
    return k


def check_selection(oracle, L, x, tau, flags, idx_g, cnt_g, inv_temp=None, label="",
                    max_exempt=None):
    """Bit-exact selections except tokens inside a tie band (tie_kinds); those
    are counted and their GPU result is checked for validity.  Outside the
    bands the kept set and count must equal the oracle's exactly, and the
    listed order too, except that experts whose logits tie within TIE_BAND
    may be listed either way.  Returns (oracle route dict, exempt mask,
    counts by kind)."""
    r = oracle.route(x, L.W_r, tau, flags=flags, bias=L.bias, inv_temp=inv_temp)
    lte = bool(flags & oracle.SELECT_LTE)
    kinds = tie_kinds(oracle, r, tau, flags)
    exempt = kinds["mass"] | kinds["cut_order"] | kinds["lte"]
    T, E = idx_g.shape
    g = r["g"]
    bad = []
    for t in range(T):
        k = int(cnt_g[t])
        assert (0 if lte else 1) <= k <= E, (t, k)
        kept = idx_g[t, :k]
        assert len(set(kept.tolist())) == k and (kept >= 0).all() and (kept < E).all(), t
        assert (idx_g[t, k:] == -1).all(), t
        if exempt[t]:
            if lte or flags & oracle.SELECT_TOPK:
                check_rule_tie_token(g[t], tau, flags, kept, oracle)
            else:
                check_tie_token(g[t], r["cum"][t], tau, flags, kept, oracle)
            continue
        ref = r["idx"][t, :r["count"][t]]
        if k != len(ref) or not (np.sort(kept) == np.sort(ref)).all():
            bad.append(t)
        elif not (kept == ref).all():
            # the same set listed in another order: only tied logits may swap
            if not kinds["prefix_order"][t] or \
                    (np.abs(g[t][kept] - g[t][ref]) > TIE_BAND).any():
                bad.append(t)
    assert not bad, "selection mismatch at tokens %s (tau=%g)" % (bad[:10], tau)
    counts = {name: int(v.sum()) for name, v in kinds.items()}
    counts["exempt"] = int(exempt.sum())
    TIE_LOG.append((label, T, float(tau), counts))
    if max_exempt is not None:
        assert counts["exempt"] <= max_exempt, \
            "%d of %d tokens exempt (%s), more than %d" % (counts["exempt"], T, counts, max_exempt)
    return r, exempt, counts


def full_size_cap(T):
    """Exempt-token cap of a full-size workload call."""
    return max(2, int(np.ceil(FULL_SIZE_EXEMPT_FRACTION * T)))


def check_output(oracle, L, x, flags, idx_g, cnt_g, y_g, g_ref, rows=None, biases=True):
    """y against the oracle evaluated on the GPU's own selection."""
    if rows is None:
        rows = np.arange(x.shape[0])
    if hasattr(L, "W_fc"):
        y_ref = oracle.mlp(x[rows], L.W_fc, L.b_fc if biases else None, L.W_proj,
                           L.b_proj if biases else None, idx_g[rows], cnt_g[rows], flags=flags,
                           g=g_ref[rows], perm=L.perm)
    else:
        y_ref = oracle.ffn(x[rows], L.W_gate, L.W_up, L.W_down, idx_g[rows], cnt_g[rows],
                           flags=flags, g=g_ref[rows], perm=L.perm)
    err = np.abs(y_g[rows].astype(np.float64) - y_ref)
    rms = float(np.sqrt(np.mean(y_ref ** 2)))
    assert np.isfinite(y_g[rows]).all()
    if rms == 0.0:  # no token kept an expert (LTE) and no output bias: y must be 0
        assert (y_g[rows] == 0).all()
        return 0.0
    worst = float(err.max()) / rms
    assert worst <= TOL, "max|dy|/RMS = %.3g" % worst
    return worst


def parity(oracle, dl, mode, x, tau, inv_temp=None, rows=None, label="", max_exempt=None):
    """One call through the C ABI checked against the oracle: selections
    (check_selection) and y on `rows` (all rows by default)."""
    idx, cnt, y = dl.run(mode, x, tau, inv_temp)
    r, exempt, counts = check_selection(oracle, dl.L, x, tau, dl.flags, idx, cnt, inv_temp,
                                        label=label or mode, max_exempt=max_exempt)
    worst = check_output(oracle, dl.L, x, dl.flags, idx, cnt, y, r["g"], rows,
                         biases=getattr(dl, "biases", True))
    return dict(idx=idx, cnt=cnt, y=y, exempt=counts["exempt"], ties=counts, worst=worst)
