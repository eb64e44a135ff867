#!/usr/bin/env python3
"""Benchmark of the PrunePath sparse-FFN forward on one MI355X.

Workload: one LLaMA-3-8B-shaped SwiGLU FFN layer (d=4096, d_ff=14336, E=112
experts of 128 neurons), decode batches T in {1, 8, 32, 64}, budget tau in
{0.5, 0.7, 0.9, 1.0}; synthetic seeded bf16 weights (N(0, 0.02^2), router
N(0, (3/sqrt(d))^2)) and tokens (N(0,1)).  A step is one call of
prunepath_ffn_decode: routing + gate/up + down for one batch, inputs resident
in HBM.  Steps rotate over several independent layer copies (> 2 GiB in
total) so that the 256 MB Infinity Cache cannot hold the weights.

Headline value: tokens/s/layer at the point selected by --T/--tau.  Each sweep
point also reports effective HBM GB/s on algorithmic bytes (router weights +
batch-union expert blocks + x + fp32 y) and its fraction of the 8 TB/s peak.
"""
import argparse
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
HBM_PEAK_GBPS = 8000.0
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "gateup_dec_llama8b_T32_tau0.7_traffic.json")


def parse_args():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--T", type=int, default=32, help="headline decode batch")
    ap.add_argument("--tau", type=float, default=0.7, help="headline budget")
    ap.add_argument("--sweep", default="full", choices=["full", "headline"],
                    help="time every (T, tau) point or only the headline one")
    ap.add_argument("--copies", type=int, default=0, help="layer copies (0 = enough for 2.2 GB)")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="target duration of the CPU-oracle timing: three single-thread and "
                         "three all-core runs share it (0 = skip the CPU leg)")
    ap.add_argument("--no-stack", action="store_true",
                    help="skip the 32-layer stacked decode measurement")
    ap.add_argument("--no-prefill", action="store_true",
                    help="skip the 2048-token prefill measurement")
    ap.add_argument("--no-mlp", action="store_true",
                    help="skip the GPT-2 Medium (non-gated GELU MLP) decode leg")
    ap.add_argument("--no-kmeans", action="store_true",
                    help="skip the balanced k-means (neuron clustering) leg")
    ap.add_argument("--no-loss", action="store_true",
                    help="skip the router-loss (training regularisers) leg")
    ap.add_argument("--no-skewed", action="store_true",
                    help="skip the wide skewed-routing layer (Qwen2-7B FFN shape)")
    ap.add_argument("--no-rules", action="store_true",
                    help="skip the comparison selection rules (strict, top-k, LTE)")
    ap.add_argument("--calibrate-copy-mib", type=int, default=0,
                    help="also run a plain device copy of this many MiB (5 times), the "
                         "reference dispatch for scaling HBM byte counters")
    return ap.parse_args()


# The sources the decode kernels (the roofline's gateup_dec_k and its down
# projection) are built from: the committed byte counters stay valid while
# these are unchanged.
DECODE_SOURCES = ("include/prunepath.h", "paper_2605_28283_amd/csrc/pp_internal.h",
                  "paper_2605_28283_amd/csrc/pp_select.h", "paper_2605_28283_amd/csrc/pp_gateup.h",
                  "paper_2605_28283_amd/csrc/pp_decode.hip")


def source_hash():
    h = hashlib.sha256()
    for f in DECODE_SOURCES:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def device_layer(torch, d, d_ff, E, seed):
    """Another layer of the same distributions, drawn on the GPU."""
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)

    def draw(shape, std):
        return (torch.randn(shape, generator=g, device="cuda", dtype=torch.float32) * std).to(
            torch.bfloat16)

    return [draw((E, d), 3.0 / math.sqrt(d)), draw((d_ff, d), 0.02), draw((d_ff, d), 0.02),
            draw((d, d_ff), 0.02)]


def main():
    args = parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path "
              "(--gpus %d requested)." % args.gpus, file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2605_28283_amd as pp
    from paper_2605_28283_amd.workloads import WORKLOADS, workload_layer, workload_tokens

    pp.load()
    torch.cuda.init()
    dev_name = torch.cuda.get_device_name(0)
    w = WORKLOADS["llama8b_decode"]
    d, d_ff, E = w.d, w.d_ff, w.E
    layer_bytes = 3 * d_ff * d * 2 + E * d * 2
    n_copies = args.copies or max(2, math.ceil(2.2e9 / layer_bytes))
    T_max = max(w.T)
    stream = torch.cuda.current_stream()

    # ---- layers: copy 0 from the seeded numpy generator (shared with the CPU
    # baseline), the rest drawn on the GPU
    L0 = workload_layer(w, 0)
    handles = []
    for c in range(n_copies):
        if c == 0:
            Wt = [torch.from_numpy(a.view(np.int16)).cuda()
                  for a in (L0.W_r, L0.W_gate, L0.W_up, L0.W_down)]
        else:
            Wt = device_layer(torch, d, d_ff, E, 1000 + c)
        handles.append(pp.prunepath_create(d, d_ff, E, T_max, *Wt))
        del Wt
    torch.cuda.synchronize()
    torch.cuda.empty_cache()

    x_np, _ = workload_tokens(w, T_max, 0)
    x = torch.from_numpy(x_np.view(np.int16)).cuda()
    y = torch.empty((T_max, d), dtype=torch.float32, device="cuda")
    idx = torch.empty((T_max, E), dtype=torch.int32, device="cuda")
    cnt = torch.empty((T_max,), dtype=torch.int32, device="cuda")

    def step(i, T, tau):
        pp.prunepath_ffn_decode(handles[i % n_copies], x, T, tau, None, y, idx, cnt,
                                stream=stream)

    def union_stats(T, tau):
        """Per copy: |U| (batch-union experts), pairs sum_t k_t, and copy 0's
        selection (compared with the CPU oracle's in the cpu_baseline leg)."""
        out, sel0 = [], None
        for c, h in enumerate(handles):
            pp.prunepath_route(h, x, T, tau, None, idx, cnt, stream=stream)
            torch.cuda.synchronize()
            ii = idx[:T].cpu().numpy()
            cc = cnt[:T].cpu().numpy()
            if c == 0:
                sel0 = (ii.copy(), cc.copy())
            out.append((len(np.unique(ii[ii >= 0])), int(cc.sum()), int(cc.min()), int(cc.max())))
        return out, sel0

    def run_point(T, tau):
        ms, kavg = time_decode(torch, pp, handles, lambda i: step(i, T, tau), args.steps,
                               args.warmup, stream)
        us, sel0 = union_stats(T, tau)
        gpu_sel[(T, tau)] = sel0
        seq = [us[i % n_copies] for i in range(args.steps)]
        U = float(np.mean([s[0] for s in seq]))
        pairs = float(np.mean([s[1] for s in seq]))
        step_bytes = E * d * 2 + U * 6 * 128 * d + 2 * T * d + 4 * T * d
        gateup_bytes = U * 2 * 128 * d * 2 + 2 * T * d + pairs * 128 * 4
        down_bytes = U * 128 * d * 2 + pairs * 128 * 4 + 4 * T * d
        gbps = step_bytes / (ms * 1e-3) / 1e9
        return {
            "T": T, "tau": tau, "ms_per_step": ms, "tokens_per_s_layer": T / (ms * 1e-3),
            "union_experts": U, "pairs": pairs, "k_mean": pairs / T,
            "k_min": min(s[2] for s in us), "k_max": max(s[3] for s in us),
            # the paper's FFN sparsity (Sec. 4.1): 1 - mean kept experts / E
            "s_ffn": 1.0 - pairs / (T * E), "union_frac": U / E,
            "algorithmic_bytes": step_bytes, "effective_GBps": gbps,
            "frac_hbm_peak": gbps / HBM_PEAK_GBPS,
            "kernel_us": kavg,
            "gateup_bytes": gateup_bytes, "down_bytes": down_bytes,
            "gateup_GBps": (gateup_bytes / (kavg["gateup"] * 1e-6) / 1e9
                            if kavg["gateup"] else None),
            "down_GBps": (down_bytes / (kavg["down"] * 1e-6) / 1e9 if kavg["down"] else None),
        }

    gpu_sel = {}
    points = [(args.T, args.tau)]
    if args.sweep == "full":
        points = [(T, tau) for T in w.T for tau in w.taus]
        if (args.T, args.tau) not in points:
            points.append((args.T, args.tau))
    results = {}
    for T, tau in points:
        r = run_point(T, tau)
        results[(T, tau)] = r
        print("# T=%-3d tau=%.2f  %8.1f us/step  %9.0f tok/s/layer  s_FFN %.3f  |U|=%5.1f  "
              "%7.1f GB/s (%4.1f%% of peak)  gateup %.1f us (%.0f GB/s)  down %.1f us (%.0f GB/s)  "
              "route %.1f us" % (
                  T, tau, r["ms_per_step"] * 1e3, r["tokens_per_s_layer"], r["s_ffn"],
                  r["union_experts"],
                  r["effective_GBps"], 100 * r["frac_hbm_peak"], r["kernel_us"]["gateup"],
                  r["gateup_GBps"], r["kernel_us"]["down"], r["down_GBps"],
                  r["kernel_us"]["route"]), file=sys.stderr, flush=True)
    head = results[(args.T, args.tau)]

    # ---- traffic from the committed rocprofv3 counter summary, if it is current
    traffic = None
    try:
        with open(TRAFFIC_FILE) as f:
            tr = json.load(f)
        if tr.get("source_hash") == source_hash() and tr.get("T") == args.T and \
                abs(tr.get("tau", -1) - args.tau) < 1e-9:
            traffic = tr.get("hbm_bytes_per_launch")
    except (OSError, ValueError):
        pass

    roof = {"bound": "hbm", "achieved": head["gateup_GBps"], "peak": HBM_PEAK_GBPS,
            "unit": "GB/s",
            "frac": head["gateup_GBps"] / HBM_PEAK_GBPS if head["gateup_GBps"] else None,
            "traffic": traffic,
            "kernel": "gateup_dec_k (gate/up projections + SiLU product)",
            "algorithmic_bytes_per_launch": head["gateup_bytes"],
            "avg_launch_us": head["kernel_us"]["gateup"]}

    sweep = list(results.values())
    out = {
        "metric": "sparse-FFN decode tokens/s/layer",
        "value": head["tokens_per_s_layer"],
        "unit": "tokens/s/layer",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": head["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": "llama8b_ffn_decode", "d_model": d, "d_ff": d_ff, "experts": E,
                   "T": args.T, "tau": args.tau, "selection": "nucleus", "aggregation": "sum",
                   "layer_copies": n_copies, "device": dev_name},
        "effective_GBps": head["effective_GBps"],
        "frac_hbm_peak": head["frac_hbm_peak"],
        "roofline": roof,
        "cpu_baseline": None,
        "sweep": sweep,
        "source_hash": source_hash(),
    }
    for h in handles:
        pp.prunepath_destroy(h)
    handles = []
    torch.cuda.empty_cache()
    skewed = None
    if not args.no_skewed:
        skewed = bench_skewed(args, torch, np, pp)
        out["skewed"] = skewed["points"]
    if not args.no_rules:
        out["rules"] = bench_rules(args, torch, np, pp, x, n_copies)
    if not args.no_prefill:
        out["prefill"] = bench_prefill(args, torch, np, pp)
    if not args.no_stack:
        out["stack"] = bench_stack(args, torch, np, pp)
    if not args.no_mlp:
        out["gpt2m_mlp"] = bench_mlp(args, torch, np, pp)
    if not args.no_loss:
        out["router_loss"] = bench_loss(args, torch, np, pp)
    if not args.no_kmeans:
        out["kmeans"] = bench_kmeans(args, torch, np, pp)
    # ---- the CPU oracle (rank 0, N = 1), after every GPU leg
    if args.cpu_seconds > 0:
        cpu, stats = cpu_baseline_leg(args, np, L0, x_np, gpu_sel, skewed, head)
        out["cpu_baseline"] = cpu
        for r in sweep:
            r["oracle_selection"] = stats.get(("llama8b", r["T"], r["tau"]))
        if skewed:
            for r in out["skewed"]:
                r["oracle_selection"] = stats.get(("qwen7b", r["T"], r["tau"]))
    if args.calibrate_copy_mib > 0:
        n = args.calibrate_copy_mib * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        out["calibration_copy_bytes"] = 4 * n
    print(json.dumps(out), flush=True)


MFMA_BF16_PEAK_TFLOPS = 2500.0


def time_decode(torch, pp, handles, call, steps, warmup, stream):
    """Times `call(i)` (one decode step on layer copy i % len(handles)) over
    `steps` calls after `warmup`, then repeats the calls with per-kernel HIP
    events recorded on the call stream.  Returns (ms per step, average
    microseconds per launch by kernel kind)."""
    for i in range(warmup):
        call(i)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for i in range(steps):
        call(i)
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    for h in handles:
        pp.prunepath_profile_begin(h, 4 * steps)
    for i in range(steps):
        call(i)
    torch.cuda.synchronize()
    kms = [0.0] * pp.PP_KERNEL_COUNT
    kn = [0] * pp.PP_KERNEL_COUNT
    for h in handles:
        a, n = pp.prunepath_profile_end(h)
        kms = [u + v for u, v in zip(kms, a)]
        kn = [u + v for u, v in zip(kn, n)]
    kavg = {name: (kms[k] / kn[k] * 1e3 if kn[k] else None)
            for name, k in (("route", pp.PP_KERNEL_ROUTE), ("gateup", pp.PP_KERNEL_GATEUP),
                            ("down", pp.PP_KERNEL_DOWN))}
    return ms, kavg


def bench_skewed(args, torch, np, pp):
    """The wide skewed-routing layer: the Qwen2-7B FFN shape (d 3584, d_ff
    18944, E 148 experts of 128), router logits (W_r x + b) / temperature
    with b ~ Gumbel(0, 1.5) per expert and temperature ~ U(0.5, 2) per token,
    decode T = 64, tau in {0.5, 0.9}.  Calls rotate over 6 layer copies
    (2.4 GB) drawn on the GPU, each with its own bias draw; the tokens and
    temperatures are the seeded workload's.  Algorithmic bytes as for the
    main sweep plus the bias and temperatures."""
    from paper_2605_28283_amd.workloads import WORKLOADS, workload_tokens
    w = WORKLOADS["qwen7b_skewed"]
    d, d_ff, E, T = w.d, w.d_ff, w.E, w.T[0]
    layer_bytes = 3 * d_ff * d * 2 + E * d * 2
    ncp = max(2, math.ceil(2.2e9 / layer_bytes))
    hs, bts = [], []
    Wr0 = bias0 = None
    for c in range(ncp):
        Wt = device_layer(torch, d, d_ff, E, 5000 + c)
        b = np.random.default_rng(5000 + c).gumbel(0.0, 1.5, size=E).astype(np.float32)
        bts.append(torch.from_numpy(b).cuda())
        hs.append(pp.prunepath_create(d, d_ff, E, T, *Wt, router_bias=bts[-1]))
        if c == 0:
            Wr0 = Wt[0].view(torch.int16).cpu().numpy().view(np.uint16)
            bias0 = b
        del Wt
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    x_np, it_np = workload_tokens(w, T, 0)
    x = torch.from_numpy(x_np.view(np.int16)).cuda()
    it = torch.from_numpy(it_np).cuda()
    y = torch.empty((T, d), dtype=torch.float32, device="cuda")
    idx = torch.empty((T, E), dtype=torch.int32, device="cuda")
    cnt = torch.empty((T,), dtype=torch.int32, device="cuda")
    stream = torch.cuda.current_stream()
    planned = {0.5: 146e6, 0.9: 376e6}  # simulated union bytes of this workload's distributions
    res, sel = [], {}
    for tau in w.taus:
        ms, kavg = time_decode(
            torch, pp, hs,
            lambda i: pp.prunepath_ffn_decode(hs[i % ncp], x, T, tau, it, y, idx, cnt,
                                              stream=stream),
            args.steps, args.warmup, stream)
        us, ks = [], []
        for c, h in enumerate(hs):
            pp.prunepath_route(h, x, T, tau, it, idx, cnt, stream=stream)
            torch.cuda.synchronize()
            ii, cc = idx.cpu().numpy(), cnt.cpu().numpy()
            if c == 0:
                sel[tau] = (ii.copy(), cc.copy())
            us.append(len(np.unique(ii[ii >= 0])))
            ks.append(cc)
        seq = [i % ncp for i in range(args.steps)]
        U = float(np.mean([us[i] for i in seq]))
        pairs = float(np.mean([ks[i].sum() for i in seq]))
        nbytes = E * d * 2 + 4 * E + U * 6 * 128 * d + 2 * T * d + 4 * T + 4 * T * d
        gbps = nbytes / (ms * 1e-3) / 1e9
        gu_bytes = U * 2 * 128 * d * 2 + 2 * T * d + pairs * 128 * 4
        dn_bytes = U * 128 * d * 2 + pairs * 128 * 4 + 4 * T * d
        r = {"workload": "qwen7b_skewed_decode", "d_model": d, "d_ff": d_ff, "experts": E,
             "T": T, "tau": tau, "layer_copies": ncp, "ms_per_step": ms,
             "tokens_per_s_layer": T / (ms * 1e-3), "union_experts": U,
             "union_frac": U / E, "pairs": pairs, "k_mean": pairs / T,
             "k_min": int(min(k.min() for k in ks)), "k_max": int(max(k.max() for k in ks)),
             "s_ffn": 1.0 - pairs / (T * E), "algorithmic_bytes": nbytes,
             "effective_GBps": gbps, "frac_hbm_peak": gbps / HBM_PEAK_GBPS,
             "planned_bytes": planned.get(tau),
             "planned_ideal_us": planned[tau] / (HBM_PEAK_GBPS * 1e3) if tau in planned else None,
             "kernel_us": kavg,
             "gateup_GBps": gu_bytes / (kavg["gateup"] * 1e-6) / 1e9 if kavg["gateup"] else None,
             "down_GBps": dn_bytes / (kavg["down"] * 1e-6) / 1e9 if kavg["down"] else None}
        res.append(r)
        print("# skewed qwen7b T=%d tau=%.2f  %7.1f us/step  %9.0f tok/s/layer  k %.2f (%d..%d)  "
              "s_FFN %.3f  |U| %.1f of %d  %7.1f GB/s (%4.1f%% of peak)  gateup %.1f us  down "
              "%.1f us  route %.1f us" % (
                  T, tau, ms * 1e3, r["tokens_per_s_layer"], r["k_mean"], r["k_min"], r["k_max"],
                  r["s_ffn"], U, E, gbps, 100 * gbps / HBM_PEAK_GBPS, kavg["gateup"],
                  kavg["down"], kavg["route"]), file=sys.stderr, flush=True)
    for h in hs:
        pp.prunepath_destroy(h)
    torch.cuda.empty_cache()
    return {"points": res, "sel": sel, "W_r0": Wr0, "bias0": bias0, "x": x_np, "inv_temp": it_np}


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def selection_stats(oracle, np, r, idx, cnt, tau):
    """The GPU's selections against the oracle's fp64 routing r: tokens in
    the tie bands (cumulative mass within 1e-5 of tau; last kept and first
    dropped logits within 1e-5) and tokens whose kept set, count or order
    differs outside them (order may differ only between tied logits)."""
    near = oracle.near_tie(r["cum"], tau)
    cut = oracle.cut_order_tie(r["g"], r["count"])
    pre = oracle.prefix_order_tie(r["g"], r["count"])
    ex = near | cut
    bad = 0
    for t in range(len(cnt)):
        if ex[t]:
            continue
        k = int(cnt[t])
        ref = r["idx"][t, :r["count"][t]]
        kept = idx[t, :k]
        if k != len(ref) or not (np.sort(kept) == np.sort(ref)).all():
            bad += 1
        elif not (kept == ref).all() and not pre[t]:
            bad += 1
    return {"tokens": int(len(cnt)), "near_tie": int(near.sum()), "cut_tie": int(cut.sum()),
            "order_only_ties": int(pre.sum()), "exempt": int(ex.sum()),
            "mismatch_outside_bands": bad}


def cpu_baseline_leg(args, np, L0, x_np, gpu_sel, skewed, head):
    """Everything that runs the CPU oracle.  (1) Its throughput on the
    headline batch (layer copy 0, T = --T, tau = --tau, route + kept-expert
    FFN in fp64), three runs single-threaded and three on all the threads
    OpenMP is given, each figure the median of its three; (2) for every
    decode point timed above, the oracle's routing of layer copy 0 (and of
    the skewed leg's copy 0) against the GPU's selection of the same batch."""
    import oracle
    T, tau = args.T, args.tau
    xs = x_np[:T]

    def one():
        oracle.forward(xs, L0.W_r, L0.W_gate, L0.W_up, L0.W_down, tau)

    all_threads = oracle.num_threads()
    per_run = args.cpu_seconds / 6.0

    def three_runs(threads):
        oracle.set_num_threads(threads)
        one()  # warm: library load, page-in of the weights
        t0 = time.perf_counter()
        one()
        n = max(1, int(round(per_run / (time.perf_counter() - t0))))
        rates = []
        for _ in range(3):
            t0 = time.perf_counter()
            for _ in range(n):
                one()
            rates.append(n * T / (time.perf_counter() - t0))
        return rates, n

    single, n1 = three_runs(1)
    multi, nm = three_runs(all_threads)
    oracle.set_num_threads(all_threads)
    med1, medm = float(np.median(single)), float(np.median(multi))
    gpu = head["tokens_per_s_layer"]
    cpu = {"value": medm, "unit": "tokens/s/layer", "cores": all_threads, "kind": "oracle",
           "sample": "fp64 C oracle (route + kept-expert FFN), LLaMA-3-8B layer copy 0, the "
                     "T=%d headline batch at tau=%g: median of 3 runs of %d calls on %d "
                     "threads (single-thread: median of 3 runs of %d calls)" % (
                         T, tau, nm, all_threads, n1),
           "runs": multi,
           "single_thread": {"value": med1, "cores": 1, "runs": single},
           "nproc": os.cpu_count(),
           "affinity_cpus": len(os.sched_getaffinity(0)),
           "cpu_model": cpu_model(),
           "gpu_speedup_vs_all_threads": gpu / medm,
           "gpu_speedup_vs_single_thread": gpu / med1}
    print("# CPU oracle (%s, nproc %s): %.0f tokens/s/layer on %d threads, %.0f single-threaded "
          "(GPU %.0fx / %.0fx)" % (cpu["cpu_model"], cpu["nproc"], medm, all_threads, med1,
                                   gpu / medm, gpu / med1), file=sys.stderr, flush=True)
    stats = {}
    for (Tp, taup), (ii, cc) in gpu_sel.items():
        r = oracle.route(x_np[:Tp], L0.W_r, taup)
        stats[("llama8b", Tp, taup)] = selection_stats(oracle, np, r, ii, cc, taup)
    if skewed:
        for taup, (ii, cc) in skewed["sel"].items():
            r = oracle.route(skewed["x"], skewed["W_r0"], taup, bias=skewed["bias0"],
                             inv_temp=skewed["inv_temp"])
            stats[("qwen7b", len(cc), taup)] = selection_stats(oracle, np, r, ii, cc, taup)
    bad = sum(v["mismatch_outside_bands"] for v in stats.values())
    ties = sum(v["exempt"] for v in stats.values())
    print("# oracle selections: %d decode points, %d tokens in tie bands, %d mismatches outside "
          "them" % (len(stats), ties, bad), file=sys.stderr, flush=True)
    return cpu, stats


def bench_rules(args, torch, np, pp, x, n_copies):
    """The selection rules beside the default nucleus cut, on the same
    LLaMA-3-8B decode workload (T=32, layer copies drawn on the GPU):
    the printed strict rule at tau=0.7, forced top-4, and LTE's sigmoid
    threshold delta=0.95."""
    from paper_2605_28283_amd.workloads import WORKLOADS
    w = WORKLOADS["llama8b_decode"]
    d, d_ff, E, T = w.d, w.d_ff, w.E, args.T
    res = []
    for name, flags, p in (("strict", pp.PP_SELECT_STRICT, 0.7), ("topk", pp.PP_SELECT_TOPK, 4.0),
                           ("lte", pp.PP_SELECT_LTE, 0.95)):
        hs = []
        for c in range(n_copies):
            Wt = device_layer(torch, d, d_ff, E, 3000 + c)
            hs.append(pp.prunepath_create(d, d_ff, E, T, *Wt, flags=flags))
            del Wt
        torch.cuda.synchronize()
        y = torch.empty((T, d), dtype=torch.float32, device="cuda")
        idx = torch.empty((T, E), dtype=torch.int32, device="cuda")
        cnt = torch.empty((T,), dtype=torch.int32, device="cuda")
        stream = torch.cuda.current_stream()
        for i in range(args.warmup):
            pp.prunepath_ffn_decode(hs[i % n_copies], x, T, p, None, y, idx, cnt, stream=stream)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for i in range(args.steps):
            pp.prunepath_ffn_decode(hs[i % n_copies], x, T, p, None, y, idx, cnt, stream=stream)
        e1.record(stream)
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / args.steps
        ks, us = [], []
        for h in hs:
            pp.prunepath_route(h, x, T, p, None, idx, cnt, stream=stream)
            torch.cuda.synchronize()
            ii = idx[:T].cpu().numpy()
            ks.append(float(cnt[:T].float().mean().item()))
            us.append(len(np.unique(ii[ii >= 0])))
        for h in hs:
            pp.prunepath_destroy(h)
        torch.cuda.empty_cache()
        U = float(np.mean(us))
        nbytes = E * d * 2 + U * 6 * 128 * d + 6 * T * d
        r = {"rule": name, "param": p, "T": T, "ms_per_step": ms,
             "tokens_per_s_layer": T / (ms * 1e-3), "k_mean": float(np.mean(ks)),
             "union_experts": U, "effective_GBps": nbytes / (ms * 1e-3) / 1e9}
        res.append(r)
        print("# rule %-6s %5.2f  T=%d  %8.1f us/step  %9.0f tok/s/layer  k %.2f  |U| %.1f  %7.1f GB/s"
              % (name, p, T, ms * 1e3, r["tokens_per_s_layer"], r["k_mean"], U,
                 r["effective_GBps"]), file=sys.stderr, flush=True)
    return res


def bench_prefill(args, torch, np, pp):
    """One LLaMA-3-8B-shaped layer, T=2048 prefill (rows scaled by
    LogNormal(0, 0.5)), tau in {0.7, 0.9}; calls rotate over 3 layer copies
    (1.06 GB) so the Infinity Cache cannot hold the weights.  Reports MFMA
    utilisation on algorithmic flops (router 2*E*d*T + 6*128*d*sum_t k_t)
    against the dense bf16 peak, beside the attainable roofline
    min(peak, HBM peak x algorithmic intensity)."""
    from paper_2605_28283_amd.workloads import WORKLOADS, workload_tokens
    w = WORKLOADS["llama8b_prefill"]
    d, d_ff, E, T = w.d, w.d_ff, w.E, w.T[0]
    handles = []
    for c in range(3):
        Wt = device_layer(torch, d, d_ff, E, 2000 + c)
        handles.append(pp.prunepath_create(d, d_ff, E, T, *Wt))
        del Wt
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    x_np, _ = workload_tokens(w, T, 0)
    x = torch.from_numpy(x_np.view(np.int16)).cuda()
    y = torch.empty((T, d), dtype=torch.float32, device="cuda")
    idx = torch.empty((T, E), dtype=torch.int32, device="cuda")
    cnt = torch.empty((T,), dtype=torch.int32, device="cuda")
    stream = torch.cuda.current_stream()
    steps = max(5, args.steps // 10)
    res = []
    for tau in w.taus:
        for i in range(3):
            pp.prunepath_ffn_prefill(handles[i % 3], x, T, tau, None, y, idx, cnt, stream=stream)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for i in range(steps):
            pp.prunepath_ffn_prefill(handles[i % 3], x, T, tau, None, y, idx, cnt, stream=stream)
        e1.record(stream)
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / steps
        for h in handles:
            pp.prunepath_profile_begin(h, 8 * steps)
        for i in range(steps):
            pp.prunepath_ffn_prefill(handles[i % 3], x, T, tau, None, y, idx, cnt, stream=stream)
        torch.cuda.synchronize()
        kms = [0.0] * pp.PP_KERNEL_COUNT
        for h in handles:
            a, _ = pp.prunepath_profile_end(h)
            kms = [u + v for u, v in zip(kms, a)]
        kus = {name: kms[k] / steps * 1e3 for name, k in (
            ("route", pp.PP_KERNEL_ROUTE), ("dispatch", pp.PP_KERNEL_DISPATCH),
            ("gateup", pp.PP_KERNEL_GATEUP), ("down", pp.PP_KERNEL_DOWN))}
        ks = []
        for h in handles:
            pp.prunepath_route(h, x, T, tau, None, idx, cnt, stream=stream)
            torch.cuda.synchronize()
            ks.append(int(cnt.sum().item()))
        pairs = float(np.mean(ks))
        flops = 2.0 * E * d * T + 6.0 * 128 * d * pairs
        nbytes = E * d * 2 + E * 6 * 128 * d + 2 * T * d + 4 * T * d
        tflops = flops / (ms * 1e-3) / 1e12
        attainable = min(MFMA_BF16_PEAK_TFLOPS, HBM_PEAK_GBPS * 1e-3 * flops / nbytes)
        res.append({"T": T, "tau": tau, "ms_per_call": ms, "tokens_per_s": T / (ms * 1e-3),
                    "k_mean": pairs / T, "algorithmic_tflop": flops / 1e12,
                    "achieved_tflops": tflops, "mfma_util": tflops / MFMA_BF16_PEAK_TFLOPS,
                    "attainable_tflops": attainable, "frac_attainable": tflops / attainable,
                    "effective_GBps": nbytes / (ms * 1e-3) / 1e9, "kernel_us": kus})
        print("# prefill T=%d tau=%.2f: %.3f ms/call, %.0f tokens/s, k %.2f, %.1f TFLOP/s "
              "(%.1f%% of bf16 peak, %.1f%% of the attainable %.0f)  [%s]" % (
                  T, tau, ms, T / (ms * 1e-3), pairs / T, tflops, 100 * tflops / MFMA_BF16_PEAK_TFLOPS,
                  100 * tflops / attainable, attainable,
                  " ".join("%s %.1f us" % kv for kv in kus.items())), file=sys.stderr, flush=True)
    for h in handles:
        pp.prunepath_destroy(h)
    torch.cuda.empty_cache()
    return res


def bench_stack(args, torch, np, pp):
    """32 LLaMA-3-8B-shaped layers chained by residual + RMSNorm, decode T=16,
    tau=0.8, one step = all 32 layers, captured once in a HIP graph and
    replayed; 11.3 GB of distinct weights per step, so no cache holds them."""
    from paper_2605_28283_amd.stack import DecodeStack
    from paper_2605_28283_amd.workloads import (WORKLOADS, bf16_to_f32, make_layer_device,
                                                stack_layer_seed, workload_tokens)
    w = WORKLOADS["llama8b_stack32"]
    d, E, T, tau = w.d, w.E, w.T[0], w.taus[0]
    handles = []
    for l in range(w.layers):
        W = make_layer_device(w.d, w.d_ff, w.E, stack_layer_seed(l))
        handles.append(pp.prunepath_create(w.d, w.d_ff, w.E, T, W["W_r"], W["W_gate"],
                                           W["W_up"], W["W_down"]))
        del W
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    S = DecodeStack(handles, d, E, T, tau)
    x0_bits, _ = workload_tokens(w, T)
    S.set_input(torch.from_numpy(bf16_to_f32(x0_bits).copy()).cuda())
    for _ in range(3):
        S.enqueue()
    torch.cuda.synchronize()
    S.capture()
    steps = max(5, args.steps // 10)
    for _ in range(3):
        S.replay()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(steps):
        S.replay()
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    cnt = S.cnt.cpu().numpy()
    idx = S.idx.cpu().numpy()
    union = [int(len(np.unique(idx[l][idx[l] >= 0]))) for l in range(w.layers)]
    layer_bytes = [E * d * 2 + u * 6 * 128 * d + 2 * T * d + 4 * T * d + 14 * T * d
                   for u in union]
    hist = np.bincount(cnt.ravel(), minlength=E + 1)
    for h in handles:
        pp.prunepath_destroy(h)
    gbps = sum(layer_bytes) / (ms * 1e-3) / 1e9
    print("# stack32 T=%d tau=%.2f: %.3f ms/step (%.1f us/layer), %.0f tokens/s, "
          "mean k %.2f, mean |U| %.1f, %.0f GB/s" % (T, tau, ms, ms * 1e3 / w.layers,
                                                    T / (ms * 1e-3), cnt.mean(),
                                                    np.mean(union), gbps),
          file=sys.stderr, flush=True)
    return {"workload": "llama8b_stack32_decode", "layers": w.layers, "T": T, "tau": tau,
            "graph": True, "steps": steps, "ms_per_step": ms,
            "us_per_layer": ms * 1e3 / w.layers, "tokens_per_s": T / (ms * 1e-3),
            "tokens_per_s_layer": T / (ms * 1e-3 / w.layers),
            "algorithmic_bytes_per_step": float(sum(layer_bytes)),
            "effective_GBps": gbps, "frac_hbm_peak": gbps / HBM_PEAK_GBPS,
            "k_mean_per_layer": [float(v) for v in cnt.mean(axis=1)],
            "union_per_layer": union,
            "k_histogram": {str(k): int(v) for k, v in enumerate(hist) if v}}


def bench_mlp(args, torch, np, pp):
    """The paper's GPT-2 Medium target: one non-gated GELU MLP layer with
    biases (d 1024, d_ff 4096, E 32 experts of 128), decode T in {1, 32},
    tau in {0.7, 0.9, 1.0}.  Calls rotate over 24 layer copies (384 MB of
    weights, the whole model's MLPs, more than the Infinity Cache holds).
    Algorithmic bytes: router E d 2 + union experts x (W_fc + W_proj 4 x 128 d,
    b_fc 512) + b_proj 4 d + tokens 2 T d + y 4 T d."""
    from paper_2605_28283_amd.workloads import WORKLOADS, make_mlp_layer, workload_tokens
    w = WORKLOADS["gpt2m_decode"]
    d, d_ff, E, ncp = w.d, w.d_ff, w.E, 24
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    hs = []
    for c in range(ncp):
        L = make_mlp_layer(d, d_ff, E, 4000 + c)
        hs.append(pp.prunepath_create_mlp(d, d_ff, E, 64, dev(L.W_r.view(np.int16)),
                                          dev(L.W_fc.view(np.int16)), dev(L.b_fc),
                                          dev(L.W_proj.view(np.int16)), dev(L.b_proj)))
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    res = []
    for T in (1, 32):
        xb, _ = workload_tokens(w, T)
        x = dev(xb.view(np.int16))
        y = torch.empty((T, d), dtype=torch.float32, device="cuda")
        idx = torch.empty((T, E), dtype=torch.int32, device="cuda")
        cnt = torch.empty((T,), dtype=torch.int32, device="cuda")
        for tau in (0.7, 0.9, 1.0):
            for i in range(args.warmup):
                pp.prunepath_ffn_decode(hs[i % ncp], x, T, tau, None, y, idx, cnt, stream=stream)
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            for i in range(args.steps):
                pp.prunepath_ffn_decode(hs[i % ncp], x, T, tau, None, y, idx, cnt, stream=stream)
            e1.record(stream)
            torch.cuda.synchronize()
            ms = e0.elapsed_time(e1) / args.steps
            us, ks = [], []
            for h in hs:
                pp.prunepath_route(h, x, T, tau, None, idx, cnt, stream=stream)
                torch.cuda.synchronize()
                ii = idx.cpu().numpy()
                us.append(len(np.unique(ii[ii >= 0])))
                ks.append(float(cnt.float().mean().item()))
            U = float(np.mean(us))
            nbytes = E * d * 2 + U * (4 * 128 * d + 512) + 4 * d + 6 * T * d
            gbps = nbytes / (ms * 1e-3) / 1e9
            r = {"T": T, "tau": tau, "ms_per_step": ms, "tokens_per_s_layer": T / (ms * 1e-3),
                 "k_mean": float(np.mean(ks)), "union_experts": U,
                 "algorithmic_bytes": nbytes, "effective_GBps": gbps,
                 "frac_hbm_peak": gbps / HBM_PEAK_GBPS}
            res.append(r)
            print("# gpt2m MLP T=%-2d tau=%.2f  %7.1f us/step  %9.0f tok/s/layer  k %.2f  |U| %.1f"
                  "  %6.0f GB/s" % (T, tau, ms * 1e3, r["tokens_per_s_layer"], r["k_mean"], U,
                                     gbps), file=sys.stderr, flush=True)
    for h in hs:
        pp.prunepath_destroy(h)
    torch.cuda.empty_cache()
    return {"workload": "gpt2m_mlp_decode", "d": d, "d_ff": d_ff, "experts": E,
            "layer_copies": ncp, "points": res}


def bench_kmeans(args, torch, np, pp):
    """MoEfication's clustering at the LLaMA-3-8B split: the d_ff = 14336
    neuron rows of D = 4096 (bf16, planted structure: centres N(0, 0.02^2)
    plus N(0, 0.02^2) noise) into E = 112 balanced clusters of 128, 5 Lloyd
    iterations from seeded initial rows, timed as one call (it blocks).
    Reports ms per iteration, auction rounds per assignment, and the distance
    GEMM's byte and flop rates (F read once, 3 bf16 MFMA passes)."""
    import time
    from paper_2605_28283_amd.workloads import bf16_to_f32, make_clustered_features
    n, D, k, iters = 14336, 4096, 112, 5
    F_bits, _, init_rows = make_clustered_features(n, D, k, 0)
    F = torch.from_numpy(F_bits.view(np.int16)).cuda()
    init = torch.from_numpy(bf16_to_f32(F_bits)[init_rows].copy()).cuda()
    ws = torch.empty(pp.prunepath_kmeans_workspace(n, D, k), dtype=torch.uint8, device="cuda")
    assign = torch.empty(n, dtype=torch.int32, device="cuda")
    perm = torch.empty(n, dtype=torch.int32, device="cuda")
    cent = torch.empty((k, D), dtype=torch.float32, device="cuda")
    obj = torch.empty(iters, dtype=torch.float32, device="cuda")
    pp.prunepath_balanced_kmeans(F, n, D, k, init, 1, assign, perm, cent, ws)  # warm-up
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    rounds = pp.prunepath_balanced_kmeans(F, n, D, k, init, iters, assign, perm, cent, ws,
                                          objective=obj)
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3
    o = obj.cpu().numpy().tolist()
    print("# kmeans n=%d D=%d k=%d: %.2f ms for %d iterations (%.2f ms/iter), rounds %s, "
          "objective %.4g -> %.4g" % (n, D, k, ms, iters, ms / iters, rounds, o[0], o[-1]),
          file=sys.stderr, flush=True)
    return {"workload": "kmeans_llama8b_dff14336_E112", "n": n, "D": D, "k": k, "iters": iters,
            "ms_total": ms, "ms_per_iter": ms / iters, "rounds": rounds, "objective": o,
            "dist_gemm_bytes": 2.0 * n * D, "dist_gemm_bf16_flops": 3 * 2.0 * n * k * D}


def bench_loss(args, torch, np, pp):
    """Routing regularisers forward + backward over a training batch of
    B = 16384 logit rows, E = 112 (eta 0.5, lambda 0.05, gamma 0.1, eps 1e-8).
    Calls rotate over 48 logit/gradient buffer pairs (700 MB), more than the
    Infinity Cache holds, captured once in a HIP graph and replayed.
    Algorithmic bytes: g read twice, dg written once, 12 B E per call."""
    from paper_2605_28283_amd.workloads import ROUTER_LOSS_B, ROUTER_LOSS_E, make_router_logits
    B, E, ncp = ROUTER_LOSS_B, ROUTER_LOSS_E, 48
    g0 = torch.from_numpy(make_router_logits(B, E, 0)).cuda()
    gs = [g0 + 0.01 * c for c in range(ncp)]
    dgs = [torch.empty_like(g0) for _ in range(ncp)]
    ws = torch.empty(pp.prunepath_router_loss_workspace(B, E) // 4, dtype=torch.float32,
                     device="cuda")
    losses = torch.empty(4, dtype=torch.float32, device="cuda")
    # one HIP graph holds one call per buffer pair, so the timing sees the
    # kernels and their boundaries, not the Python launch rate
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        for c in range(ncp):
            pp.prunepath_router_loss(gs[c], B, E, 1e-8, 0.5, 0.05, 0.1, losses, dgs[c], ws,
                                     stream=side)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        for c in range(ncp):
            pp.prunepath_router_loss(gs[c], B, E, 1e-8, 0.5, 0.05, 0.1, losses, dgs[c], ws,
                                     stream=torch.cuda.current_stream())
    stream = torch.cuda.current_stream()
    reps = max(2, args.steps // ncp)
    for _ in range(max(1, args.warmup // ncp)):
        graph.replay()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(reps):
        graph.replay()
    e1.record(stream)
    torch.cuda.synchronize()
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0.record(stream)
    for i in range(args.steps):
        pp.prunepath_router_loss(gs[i % ncp], B, E, 1e-8, 0.5, 0.05, 0.1, losses, dgs[i % ncp], ws,
                                 stream=stream)
    t1.record(stream)
    torch.cuda.synchronize()
    eager = t0.elapsed_time(t1) / args.steps
    ms = e0.elapsed_time(e1) / (reps * ncp)
    nbytes = 12.0 * B * E
    gbps = nbytes / (ms * 1e-3) / 1e9
    print("# router loss fwd+bwd B=%d E=%d: %.1f us/call in a graph (%.1f us eager), "
          "%.0f GB/s (%.1f%% of HBM peak)" % (B, E, ms * 1e3, eager * 1e3, gbps,
                                              100 * gbps / HBM_PEAK_GBPS),
          file=sys.stderr, flush=True)
    return {"workload": "router_loss_llama8b_B16384", "B": B, "E": E, "ms_per_call": ms,
            "us_per_call": ms * 1e3, "rows_per_s": B / (ms * 1e-3),
            "algorithmic_bytes": nbytes, "effective_GBps": gbps,
            "frac_hbm_peak": gbps / HBM_PEAK_GBPS, "launches": 3, "graph": True,
            "us_per_call_eager": eager * 1e3}


if __name__ == "__main__":
    main()
