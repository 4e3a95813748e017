"""Decode-step throughput of the ASR-KF-EGR hot path on one MI355X.

A step is the whole path for every layer and sequence: append, attention over
the active cache with relevance and the freeze schedule (one launch per layer)
plus the split combine, then entropy, recovery and the rebuild of every
active list.  Inputs are synthetic (seeded generator, device twin) and sit in
HBM before the timed region starts.

Prints one JSON line.  value = attended (active) KV token-layers per second,
from a timed loop without instrumentation; the attention kernel's duration for
the roofline comes from a replay of the same steps in which every attention
dispatch records HIP events, the per-step series from two more replays (GPU
time per step from events between steps, attended token-layers per step).
"""
import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0
WORKLOADS = {"32layer": "llama8b_32layer", "1layer": "llama8b_1layer", "ragged": "ragged",
             "recovery": "recovery_stress"}


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=112)
    ap.add_argument("--warmup", type=int, default=16)
    ap.add_argument("--workload", choices=sorted(WORKLOADS), default="32layer")
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="budget of the oracle sample (0 disables the cpu_baseline leg)")
    ap.add_argument("--relevance", choices=["abs", "softmax"], default=None,
                    help="relevance reading (default: the workload's, Eq. 2 |q.k|)")
    ap.add_argument("--scope", choices=["layer", "token"], default=None,
                    help="token-state scope (default: per layer and sequence)")
    ap.add_argument("--history-W", type=int, default=None, help="detection-count window (0 = all)")
    ap.add_argument("--candidates", choices=["outside", "inside"], default=None,
                    help="freeze candidates relative to the K-recent window (default: outside)")
    ap.add_argument("--graph", action="store_true",
                    help="time the steps as HIP graph replays: each timed step (every layer's "
                         "decode_step and the restore) is captured beforehand as a graph")
    ap.add_argument("--layers", type=int, default=0,
                    help="run only the first N layers of the workload (counter runs); 0 = all")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="BYTES",
                    help="after the run, one plain device copy of BYTES (counter calibration)")
    ap.add_argument("--summarize-trace", metavar="TRACE_DIR",
                    help="print, from a rocprofv3 --kernel-trace --stats run of this bench (same "
                         "--steps, --warmup and --layers), the kernel table and the attention "
                         "kernel's mean duration over the measured steps of each pass; no GPU work")
    ap.add_argument("--summarize-counters", nargs=3, metavar=("FETCH_DIR", "WRITE_DIR", "BENCH_LOG"),
                    help="print the HBM traffic per attention launch from two rocprofv3 --pmc "
                         "runs (FETCH_SIZE, WRITE_SIZE) made with --copy-calibration, and its "
                         "ratio to the algorithmic bytes in the JSON line that the FETCH_SIZE "
                         "run printed (BENCH_LOG); no GPU work")
    return ap.parse_args()


PASSES = ("rate", "steps", "kernel", "count")


def summarize_trace(trace_dir, layers, warmup, steps):
    """The kernel table of a rocprofv3 --stats run of this bench, and per pass
    (in launch order: rate, steps, kernel, count) the mean duration of the
    attention launches of the measured steps (each pass launches
    (warmup + steps) x layers of them), split at the midpoint between the
    shortest and longest launch (sparse below, dense above).  The profiler's
    own timestamps; passes with HIP events under the profiler also show the
    profiler's gaps around the dispatch, not inside it."""
    import csv
    import glob
    import statistics as st
    trace = glob.glob(os.path.join(trace_dir, "**", "*kernel_trace.csv"), recursive=True)[0]
    stats = glob.glob(os.path.join(trace_dir, "**", "*kernel_stats.csv"), recursive=True)
    out = {"kernels": []}
    if stats:
        for r in csv.DictReader(open(stats[0])):
            out["kernels"].append({"name": r["Name"], "calls": int(r["Calls"]),
                                   "avg_us": float(r["AverageNs"]) / 1e3,
                                   "share": float(r["Percentage"]) / 100})
    rows = [r for r in csv.DictReader(open(trace)) if "attention_kernel" in r["Kernel_Name"]]
    rows.sort(key=lambda r: int(r["Start_Timestamp"]))
    dur = [(int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3 for r in rows]
    per = (warmup + steps) * layers
    if len(dur) % per:
        raise SystemExit(f"{len(dur)} attention launches is not a whole number of passes of {per}")
    out["passes"] = {}
    for i in range(len(dur) // per):
        w = dur[i * per:(i + 1) * per][warmup * layers:]
        mid = (min(w) + max(w)) / 2
        sp = [x for x in w if x < mid]
        de = [x for x in w if x >= mid]
        out["passes"][PASSES[i] if i < len(PASSES) else str(i)] = {
            "launches": len(w), "avg_us": st.mean(w),
            "sparse": {"launches": len(sp), "avg_us": st.mean(sp)} if sp else None,
            "dense": {"launches": len(de), "avg_us": st.mean(de)} if de else None}
    return out


def summarize_counters(fetch_dir, write_dir, bench_log, timed, copy_bytes):
    """HBM bytes per attention launch from two rocprofv3 counter runs: the mean
    FETCH_SIZE and WRITE_SIZE (KiB per dispatch) of the last `timed` attention
    dispatches, each scaled by what the same counter read for the run's final
    plain device copy of `copy_bytes` bytes; and their ratio to the algorithmic
    bytes per launch of the same window (the bench line in bench_log)."""
    import csv
    import glob
    out = {}
    for d, counter in ((fetch_dir, "FETCH_SIZE"), (write_dir, "WRITE_SIZE")):
        path = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)[0]
        rows = [r for r in csv.DictReader(open(path)) if r["Counter_Name"] == counter]
        rows.sort(key=lambda r: int(r["Dispatch_Id"]))
        att = [float(r["Counter_Value"]) for r in rows if "attention_kernel" in r["Kernel_Name"]][-timed:]
        copy_kib = [float(r["Counter_Value"]) for r in rows if "copyBuffer" in r["Kernel_Name"]][-1]
        factor = copy_bytes / (copy_kib * 1024)
        mean = sum(att) / len(att)
        out[counter] = {"attention_kib_raw": mean, "copy_kib_raw": copy_kib, "factor": factor,
                        "bytes_per_launch": mean * 1024 * factor, "launches": len(att)}
    out["traffic_bytes_per_launch"] = round(out["FETCH_SIZE"]["bytes_per_launch"]
                                            + out["WRITE_SIZE"]["bytes_per_launch"])
    line = next(json.loads(x) for x in open(bench_log) if x.startswith("{"))
    algo = line["roofline"]["algorithmic_bytes_per_launch"]
    out["algorithmic_bytes_per_launch"] = algo
    out["traffic_per_algorithmic_byte"] = out["traffic_bytes_per_launch"] / algo
    return out


TRAFFIC_SUMMARY = os.path.join(ROOT, "profiles", "attention_traffic_llama3-8b-32layer.md")
ATTENTION_SOURCE = os.path.join(ROOT, "paper_2512_11221_amd", "csrc", "attention.hip")


def measured_traffic(workload):
    """HBM bytes per algorithmic byte of the attention kernel, from the
    committed rocprofv3 counter summary, if it was taken on this workload's
    shape and this kernel source; otherwise None.  The counter runs measure
    FETCH_SIZE + WRITE_SIZE per launch over a window of steps; dividing by the
    algorithmic bytes of the same launches gives a ratio that carries to any
    window of the same workload (the kernel reads 4096 B per attended
    token-layer plus a small fixed part per launch)."""
    import hashlib
    import re
    if not os.path.exists(TRAFFIC_SUMMARY):
        return None
    text = open(TRAFFIC_SUMMARY).read()
    fields = dict(re.findall(r"^- (\w+): `([^`]*)`", text, flags=re.M))
    with open(ATTENTION_SOURCE, "rb") as f:
        sha = hashlib.sha256(f.read()).hexdigest()
    if fields.get("workload") != workload or fields.get("attention_source_sha256") != sha:
        return None
    return float(fields["traffic_per_algorithmic_byte"]), fields


def metadata_bytes(w, W, K, attended, algo_bytes, traffic, roofline):
    """Bytes the timed steps move besides the K/V rows of attended tokens and
    the logits (the algorithmic bytes), from the kernels' access pattern:
    index lists (read by attention, written by compaction), freeze state (an
    upper bound: count read and write plus U write for every attended token),
    the compaction's scan of U over every position, q, out and the appended row
    of every (layer, sequence), and the split-K partials (written by attention,
    read by the combine; one workgroup per CU plus one slot per sequence), and
    the first-tile records of the attention ranges (resident mode, four or more
    layers: 32 list entries read and a 144-byte record written per range and
    state layer, the record read back by the attention launch).  The attention
    kernel's measured counter excess is given beside it."""
    import torch
    L, B, Hq, D = w.n_layers, w.batch, w.n_q_heads, w.head_dim
    esz = 2 if w.dtype == "bf16" else 4
    positions = L * sum(p + t for p in w.prefill for t in range(W + 1, W + K + 1))   # n_t, summed
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    parts = {
        "index_lists": 8 * attended,
        "freeze_state_upper_bound": 12 * attended,
        "compaction_scan": 4 * positions,
        "q_out_append": K * L * B * (Hq * D * esz + Hq * D * 4 + w.kv_bytes_per_token()),
        "split_partials": 2 * K * L * (cus + B) * Hq * (D + 2) * 4,
    }
    if w.spill_min_D == 0 and L >= 4:
        state_layers = 1 if w.scope == "token" else L
        parts["first_tile_records"] = K * state_layers * cus * (32 * 4 + 2 * 144)
    total = sum(parts.values())
    out = {"bytes_timed_steps": parts, "total": total, "fraction_of_algorithmic": total / algo_bytes}
    if traffic:
        out["attention_counter_excess"] = traffic / roofline["algorithmic_bytes_per_launch"] - 1.0
    return out


def regimes(w, W, K, series, bytes_per_token):
    """The timed steps split by regime.  Every prompt token starts uncounted,
    so the freezable cohort moves in lockstep: at a dense step (nearly) every
    position attends, at a sparse step (the method's operating point) the
    frozen cohort is out.  A step counts as dense when at least 90 % of the
    positions attend.
    Per regime: attended token-layers per attention launch, the launches'
    mean duration (the dispatch events of the kernel replay), that kernel's
    fraction of the HBM peak, and the whole step's fraction (algorithmic
    bytes, the logits included, over the step's GPU time from the events
    between steps)."""
    L, B = w.n_layers, w.batch
    out = {}
    for name in ("dense", "sparse"):
        idx = []
        for i, t in enumerate(range(W + 1, W + K + 1)):
            every = L * sum(p + t for p in w.prefill)          # positions n_t of every instance
            if (series["attended"][i] >= 0.9 * every) == (name == "dense"):
                idx.append(i)
        if not idx:
            out[name] = None
            continue
        tokens = sum(series["attended"][i] for i in idx)
        attn_ms = sum(series["attn_ms"][i] for i in idx)
        step_ms = sum(series["gpu_ms"][i] for i in idx)
        launch_us = 1e3 * attn_ms / (L * len(idx))
        achieved = bytes_per_token * tokens / (attn_ms / 1e3) / 1e9
        step_bytes = bytes_per_token * tokens + 4 * w.vocab * B * len(idx)
        out[name] = {"steps": len(idx), "token_layers_per_launch": tokens / (L * len(idx)),
                     "avg_launch_us": launch_us, "achieved": achieved,
                     "frac": achieved / PEAK_HBM_GBS,
                     "step_ms": step_ms / len(idx),
                     "step_frac": step_bytes / (step_ms / 1e3) / 1e9 / PEAK_HBM_GBS}
    return out


def cpu_baseline(w, budget_s):
    """The CPU oracle on a bounded sample: whole (layer, seq) instances in
    order (layer 0, sequences 0, 1, ...), every step of the run, until the time
    budget is spent."""
    import numpy as np
    import oracle
    from synth import gen
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        threads = 1
    attended, spent, inst_steps, done = 0, 0.0, 0, []
    order = [(l, b) for l in range(w.n_layers) for b in range(w.batch)]
    for (l, b) in order:
        P = w.prefill[b]
        K, V = gen.kv_rows(w, l, b, 0, P + w.steps)
        inst = oracle.Instance(K[:P], V[:P], w.window_K, w.tau, w.k_soft,
                               capacity=P + w.steps + 1, history_W=w.history_W,
                               relevance_kind=w.relevance, candidates=w.candidates)
        for t in range(1, w.steps + 1):
            q = gen.q_row(w, l, b, t)
            t0 = time.perf_counter()
            rec = inst.step(q, K[P + t - 1], V[P + t - 1])
            spent += time.perf_counter() - t0
            attended += len(rec.active)
            inst_steps += 1
            if spent >= budget_s:
                break
        done.append((l, b, t))
        if spent >= budget_s:
            break
    instances = len(order)
    what = ", ".join(f"layer {l} seq {b} steps 1..{t}" for l, b, t in done)
    return {"value": attended / spent, "unit": "active KV token-layers/s", "cores": threads,
            "kind": "oracle",
            "sample": f"{w.name}: {what} ({attended} attended token-layers in {spent:.1f} s); "
                      f"the full step has {instances} such instances",
            "cpu_count": os.cpu_count(),
            "affinity": len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else None,
            "ms_per_step_extrapolated": 1e3 * spent / inst_steps * instances,
            "extrapolation": f"the sample's mean time per instance step x {instances} instances"}


def main():
    args = parse()
    if args.summarize_trace:
        layers = args.layers or getattr(__import__("synth.gen", fromlist=["gen"]),
                                        WORKLOADS[args.workload])().n_layers
        print(json.dumps(summarize_trace(args.summarize_trace, layers, args.warmup, args.steps),
                         indent=1))
        return
    if args.summarize_counters:
        # the measured steps of the counter runs' last pass: one attention launch per layer
        print(json.dumps(summarize_counters(*args.summarize_counters, args.steps * max(1, args.layers),
                                            args.copy_calibration or (1 << 30)), indent=1))
        return
    if args.graph and args.warmup < 1:
        print("bench.py --graph needs at least one warm-up step before the capture", file=sys.stderr)
        sys.exit(2)
    if args.gpus != 1:
        print(f"bench.py measures one GPU only: the library has no multi-GPU path "
              f"(asked for --gpus {args.gpus}).", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2512_11221_amd as A
    from synth import gen
    from synth.device import DeviceGen

    A.load()
    torch.cuda.set_device(0)
    W, K = args.warmup, args.steps
    w = getattr(gen, WORKLOADS[args.workload])(steps=W + K)
    if args.layers:
        w = w.replace(n_layers=min(args.layers, w.n_layers))
    for key in ("relevance", "scope", "history_W", "candidates"):
        if getattr(args, key) is not None:
            w = w.replace(**{key: getattr(args, key)})
    L, B, Hq, Hkv, D = w.n_layers, w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim
    tdt = torch.bfloat16 if w.dtype == "bf16" else torch.float32

    cfg = A.make_config(L, B, Hq, Hkv, D, w.max_ctx, w.window_K, w.tau, w.k_soft, w.vocab,
                        entropy_spike=w.entropy_spike, conf_drop=w.conf_drop,
                        wr_last_N=w.wr_last_N, dtype=w.dtype, spill_min_D=w.spill_min_D,
                        history_W=w.history_W, relevance=w.relevance, scope=w.scope,
                        candidates=w.candidates)
    dg = DeviceGen(w)
    S = W + K
    Q = torch.empty((S, L, B, Hq, D), dtype=tdt, device="cuda")
    Kn = torch.empty((S, L, B, Hkv, D), dtype=tdt, device="cuda")
    Vn = torch.empty_like(Kn)
    LG = torch.empty((S, B, w.vocab), dtype=torch.float32, device="cuda")
    dg.q(1, S, Q)
    dg.new_kv(1, S, Kn, Vn)
    dg.logits(1, S, LG)
    out = torch.empty((L, B, Hq, D), dtype=torch.float32, device="cuda")

    ctx = A.asrkf_init(cfg)

    def run_pass(mode):
        """The context reset (the same device memory in every pass): prompt, W
        warm-up steps, then K steps measured as `mode` says:
          rate    no instrumentation; wall clock over the K steps (the value)
          steps   a HIP event between consecutive steps, no host waits inside
                  the loop (each step's GPU time)
          kernel  every attention dispatch records HIP events, no host waits
                  inside the loop (the kernel's execution time per launch)
          count   the host reads the counters after every step (attended
                  token-layers per step; nothing timed)"""
        A.asrkf_reset(ctx)
        Pmax = max(w.prefill)
        stage_k = torch.empty(Pmax * Hkv * D, dtype=tdt, device="cuda")
        stage_v = torch.empty_like(stage_k)
        for l in range(L):
            for b in range(B):
                P = w.prefill[b]
                dg.kv_rows(l, b, 0, P, stage_k, stage_v)
                A.asrkf_prefill(ctx, l, b, stage_k, stage_v, P)
        torch.cuda.synchronize()
        del stage_k, stage_v

        def step(t):
            i = t - 1
            for l in range(L):
                A.asrkf_decode_step(ctx, l, Q[i, l], Kn[i, l], Vn[i, l], out[l])
            A.asrkf_restore(ctx, LG[i], A.AUTO)

        for t in range(1, W + 1):
            step(t)
        torch.cuda.synchronize()
        if args.graph and mode in ("rate", "steps"):
            # every measured step captured beforehand as its own HIP graph (the same
            # kernels, reading that step's inputs); the loop launches the graphs in order
            graphs = []
            for t in range(W + 1, W + K + 1):
                g = torch.cuda.CUDAGraph()
                with torch.cuda.graph(g):
                    step(t)
                graphs.append(g)
            torch.cuda.synchronize()

            def step(t):                                         # noqa: F811
                graphs[t - W - 1].replay()
        A.asrkf_stats_reset(ctx)
        A.asrkf_set_timing(ctx, mode == "kernel")
        marks = [torch.cuda.Event(enable_timing=True) for _ in range(K + 1)] if mode == "steps" else []
        attended = []
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        if marks:
            marks[0].record()
        for t in range(W + 1, W + K + 1):
            step(t)
            if marks:
                marks[t - W].record()
            elif mode == "count":
                attended.append(A.asrkf_stats(ctx)["attended_total"])
        torch.cuda.synchronize()
        elapsed = time.perf_counter() - t0
        st = A.asrkf_stats(ctx)
        series = {}
        if mode == "steps":
            series["gpu_ms"] = [round(a.elapsed_time(b), 4) for a, b in zip(marks[:-1], marks[1:])]
        elif mode == "kernel":
            ms = A.asrkf_timing_series(ctx)
            assert len(ms) == K * L, (len(ms), K * L)
            series["launch_ms"] = [float(x) for x in ms]
            series["attn_ms"] = [round(float(ms[i * L:(i + 1) * L].sum()), 5) for i in range(K)]
        elif mode == "count":
            series["attended"] = [c - p for c, p in zip(attended, [0] + attended[:-1])]
        return elapsed, st, series

    # The step rate comes from a pass without instrumentation.  The same steps
    # are then replayed three more times on the same context (reset in between,
    # so every pass reads and writes the same device memory): with a HIP event
    # between steps (each step's GPU time), with HIP events recorded by every
    # attention dispatch (the kernel's execution time per launch, for the
    # roofline), and with the counters read after every step (attended
    # token-layers per step).  Only the last pass waits on the host inside its
    # loop, and it times nothing.
    elapsed, st, _ = run_pass("rate")
    _, _, s_steps = run_pass("steps")
    _, st_timed, s_kernel = run_pass("kernel")
    _, st_count, s_count = run_pass("count")
    assert st_timed["attended_total"] == st["attended_total"] == st_count["attended_total"]
    assert sum(s_count["attended"]) == st["attended_total"]
    A.asrkf_destroy(ctx)
    series = {"gpu_ms": s_steps["gpu_ms"], "attended": s_count["attended"], "attn_ms": s_kernel["attn_ms"]}
    del Q, Kn, Vn, LG, out

    attended = st["attended_total"]
    bytes_per_token = w.kv_bytes_per_token()          # K + V of one token, one layer
    algo_bytes = bytes_per_token * attended + 4 * w.vocab * B * K
    attn_s = st_timed["attn_kernel_ms"] / 1e3
    achieved = bytes_per_token * attended / attn_s / 1e9
    default_path = (w.relevance == "abs" and w.scope == "layer" and not w.history_W
                    and not w.spill_min_D and w.candidates == "outside")
    ratio = measured_traffic(w.name) if default_path else None
    launches = max(1, st_timed["attn_launches"])
    traffic = ratio[0] * bytes_per_token * attended / launches if ratio else None
    if args.copy_calibration > 0:
        src = torch.empty(args.copy_calibration, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    line = {
        "metric": "active-KV tokens/s per decode step + achieved HBM GB/s vs peak, 8B shape",
        "value": attended / elapsed,
        "unit": "active KV token-layers/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": W,
        "ms_per_step": 1e3 * elapsed / K,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic (seeded heavy-hitter generator, device twin)",
        "config": {"workload": w.name, "graph": bool(args.graph), "layers": L, "batch": B, "context": w.prefill[0]
                   if len(set(w.prefill)) == 1 else "ragged", "q_heads": Hq, "kv_heads": Hkv,
                   "head_dim": D, "window_K": w.window_K, "tau": w.tau, "k": w.k_soft,
                   "vocab": w.vocab, "mode": "spill" if w.spill_min_D else "resident",
                   "relevance": w.relevance, "scope": w.scope, "history_W": w.history_W,
                   "candidates": w.candidates},
        "decode_steps_per_s": K / elapsed,
        "hbm_fraction_step": algo_bytes / elapsed / 1e9 / PEAK_HBM_GBS,
        "attended_fraction": attended / max(1, sum(p + t for p in w.prefill
                                                   for t in range(W + 1, W + K + 1)) * L),
        "compression_after_run": st["compression"],
        "step_series": series,
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": achieved / PEAK_HBM_GBS, "traffic": traffic,
                     "traffic_basis": (f"HBM bytes per algorithmic byte ({ratio[0]:.4f}) from two "
                                       f"rocprofv3 counter runs (FETCH_SIZE, WRITE_SIZE, copy-"
                                       f"calibrated) of this kernel source on this workload "
                                       f"({ratio[1].get('layers', 'all')} layer(s), "
                                       f"{ratio[1].get('steps')} timed steps), times this run's "
                                       f"algorithmic bytes per launch") if ratio else None,
                     "kernel": f"attention_kernel<{w.dtype}, D={D}, G={Hq // Hkv}, Hkv={Hkv}>",
                     "algorithmic_unit": f"{bytes_per_token} B per attended token-layer (K + V rows)",
                     "launches": st_timed["attn_launches"],
                     "avg_launch_us": 1e3 * st_timed["attn_kernel_ms"] / max(1, st_timed["attn_launches"]),
                     "algorithmic_bytes_per_launch": bytes_per_token * attended
                     / max(1, st_timed["attn_launches"]),
                     "timing": "HIP events recorded by each attention dispatch, in a replay "
                               "of the same warm-up and measured steps with no host waits "
                               "inside the loop"},
    }
    line["roofline"].update(regimes(w, W, K, series, bytes_per_token))
    line["metadata"] = metadata_bytes(w, W, K, attended, algo_bytes, traffic, line["roofline"])
    if w.spill_min_D:
        row = bytes_per_token // 2                      # one K or V row
        line["spill"] = {"spill_min_D": w.spill_min_D, "rows_to_host": st["rows_to_host"],
                         "rows_from_host": st["rows_from_host"],
                         "rows_reused": st["rows_reused"],
                         "h2d_GBps": 2 * row * st["rows_from_host"] / elapsed / 1e9,
                         "d2h_GBps": 2 * row * st["rows_to_host"] / elapsed / 1e9}
    if args.cpu_seconds > 0:
        line["cpu_baseline"] = cpu_baseline(w, args.cpu_seconds)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
