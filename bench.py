#!/usr/bin/env python3
"""Decode-attention benchmark: diagonal-aware sparse vs dense on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]

One step is one decode step of the whole hot path over every layer of the
workload, all inputs resident in HBM: per layer the fused ``dsa_decode_step``
(kept-set construction, split-K attention, combine and phase-2 selection in
one pass; ``value``), and for comparison the same work as three calls
``dsa_plan -> dsa_decode_attention -> dsa_select`` (``separate_calls``).  The step is captured
once as a HIP graph and replayed (``--eager`` launches it from Python
instead).  The dense mode of the
same kernels, on the same inputs and positions, is timed alongside for the
speedup, and so are the fused steps of the sink variants of section 5.1 at
the same budget N_att (Diagonal+Sink4, and StreamingLLM: 4 sinks plus a
recent window, no selection), and the fused step over an fp8 (E4M3) copy of
the caches.  Prints one JSON line.

The default workload is the Janus-Pro-7B-like one (30 layers, 128 requests,
32 heads of d = 128), the largest model-shaped configuration on one GPU and
the model of the paper's latency breakdown (section 5.3).

``roofline`` describes the decode kernel (the dominant one): algorithmic K/V
bytes per launch (4*d bytes per attended key per KV head) divided by the
mean duration of one layer's decode on the device, from HIP events that the
extended launch binds to the start of the split-K kernel and to the end of
the last kernel of the call (the combine, when requests are split), over
``--steps`` further eager steps.  Each of
those steps waits behind a spin kernel until the host has issued all of it,
so its layers run back to back as in the timed graph replays (``--eager``
times launches as issued, without the spin).  ``cpu_baseline`` times the fp64 CPU oracle on a bounded sample
of the same workload: the C oracle on the host's cores (OpenMP over KV
heads, ``value``) and on one thread, and the Python oracle on one thread
(``--no-cpu-baseline`` skips them).
"""

from __future__ import annotations

import argparse
import copy
import hashlib
import json
import math
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
HBM_PEAK_GBPS = 8000.0
METRIC = "decode attention tokens/s + KV HBM GB/s (% of 8 TB/s), speedup vs dense"
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "decode_traffic.json")


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="janus_pro_7b")
    ap.add_argument("--positions", default=None, help="ragged | last | first")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--eager", action="store_true", help="time eager launches instead of a HIP graph")
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--only", default=None,
                    choices=["fused", "separate", "dense", "diag_sink4", "streaming", "fp8_kv",
                             "ring"],
                    help="time one step variant only (shorter profiler runs)")
    ap.add_argument("--sweep", action="store_true",
                    help="time the Janus-shaped sweep (grid x batch x window, diagonal and dense) "
                         "per layer and print one JSON line per cell instead of the step line")
    ap.add_argument("--trajectory", action="store_true",
                    help="time a whole image: every request decodes positions 0 .. H*W-1 over "
                         "every layer (fused step, and dense mode), one JSON line")
    ap.add_argument("--batch", type=int, default=0,
                    help="with --trajectory: requests per image batch instead of the workload's "
                         "(1: single-image latency)")
    ap.add_argument("--cells", default=None,
                    help="with --sweep: comma-separated substrings of the cell names to run")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MB",
                    help="run a plain device copy of MB megabytes 10 times and exit (the "
                         "reference for scaling the profiler's FETCH_SIZE/WRITE_SIZE)")
    return ap.parse_args()


KERNEL_SOURCES = ("api.hip", "decode.hip", "decode_fp8.hip", "decode_impl.h", "device.h", "internal.h")


def kernel_source_hash():
    """Hash of the decode kernels' sources and of the host code that picks
    their launch configuration (split sizes), which the committed counter
    runs depend on."""
    h = hashlib.sha256()
    for name in KERNEL_SOURCES:
        with open(os.path.join(ROOT, "paper_2609_19702_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def traffic_for(workload, src_hash):
    """HBM bytes per decode launch from committed rocprofv3 counter runs, if
    they were taken on the current kernel source."""
    try:
        with open(TRAFFIC_FILE) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    ent = rec.get(workload)
    if not ent or ent.get("kernel_hash") != src_hash:
        return None
    return ent.get("hbm_bytes_per_launch")


def oracle_units(bt, n=16):
    """A bounded sample of the workload for the CPU oracle: ``n`` requests of
    layer 0 spread over the decode positions, each with the Algorithm 1
    states its KV heads have before that position (replayed by the C
    oracle with seeded random choices), as contiguous fp64 numpy arrays."""
    import numpy as np
    import torch
    from oracle import coracle
    from paper_2609_19702_amd import synth
    w, L = bt.w, bt.layers[0]
    order = sorted(range(w.batch), key=lambda b: bt.pos_host[b])
    n = min(n, w.batch)
    pick = [order[i * (len(order) - 1) // max(n - 1, 1)] for i in range(n)]
    units = []
    qn = L.q.to(torch.float64).cpu().numpy()
    N_r, N_att = bt.p.window, bt.p.n_att
    Lp = w.prompt_len
    for b in pick:
        t = bt.pos_host[b]
        # each slice becomes one dense fp64 array in a single conversion
        arr = [x[b, :, r0:r1].to(torch.float64).contiguous().cpu().numpy()
               for x in (L.kv.k, L.kv.v) for (r0, r1) in ((0, Lp), (Lp, Lp + t + 1))]
        ints = synth.random_ints(w, 0, w.num_kv_heads * N_r, sub=b).tolist()
        heads = [coracle.replay_head(N_r, N_att, w.decode_len, t, ints[h * N_r:(h + 1) * N_r])[0]
                 for h in range(w.num_kv_heads)]
        units.append((t, np.ascontiguousarray(qn[b]), arr[0], arr[2], arr[1], arr[3], heads,
                      coracle.States.from_heads(heads, w.decode_len)))
    return pick, units


def c_oracle_loop(units, scale, seconds, threads):
    """The C oracle's decode step (attention of every head + selection, fp64)
    over ``units`` until ``seconds`` are spent inside it; returns
    (steps, seconds).  State copies are made outside the timed calls."""
    from oracle import coracle
    done, spent = 0, 0.0
    while spent < seconds:
        for (t, q, Kp, Vp, K, V, _, cstates) in units:
            st = cstates.copy()
            t0 = time.perf_counter()
            coracle.request_step(t, q, Kp, Vp, K, V, scale, "diagonal", st, threads=threads)
            spent += time.perf_counter() - t0
            done += 1
    return done, spent


def py_oracle_loop(units, scale, seconds):
    """The Python (numpy) oracle's decode step over ``units``, one thread."""
    from oracle import step as ostep
    try:
        from threadpoolctl import threadpool_limits
    except ImportError:  # pragma: no cover
        threadpool_limits = None
    ctx = threadpool_limits(1) if threadpool_limits else None
    done, spent = 0, 0.0
    try:
        while spent < seconds:
            for (t, q, Kp, Vp, K, V, heads, _) in units:
                st2 = copy.deepcopy(heads)
                t0 = time.perf_counter()
                ostep.request_step(t, q, Kp, Vp, K, V, scale, "diagonal", st2)
                spent += time.perf_counter() - t0
                done += 1
                if spent >= seconds:
                    break
    finally:
        if ctx is not None:
            ctx.__exit__(None, None, None)
    return done, spent


def cpu_baseline(bt, seconds):
    """The fp64 CPU oracle on a bounded sample (``oracle_units``): the C
    oracle with OpenMP over KV heads on the host's cores (``value``), the
    same on one thread, and the Python oracle on one thread, each decode
    step repeated until about ``seconds`` (a third of it for the Python
    oracle) is spent."""
    w = bt.w
    pick, units = oracle_units(bt)
    cores = max(1, min(16, len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity")
                       else (os.cpu_count() or 1)))
    nl = len(bt.layers)
    d_all, s_all = c_oracle_loop(units, bt.scale, seconds / 2, cores)
    d_one, s_one = c_oracle_loop(units, bt.scale, seconds / 2, 1)
    d_py, s_py = py_oracle_loop(units, bt.scale, seconds / 3)
    pos = sorted(bt.pos_host[b] for b in pick)
    return {"value": d_all / s_all / nl, "unit": "tokens/s", "cores": cores, "kind": "oracle",
            "sample": (f"C oracle (fp64, OpenMP over the {w.num_kv_heads} KV heads): one decode "
                       f"step (attention of all {w.num_q_heads} heads + phase-2 selection) of "
                       f"{len(units)} requests of layer 0 at positions {pos[0]}..{pos[-1]}, "
                       f"repeated {d_all} times in {s_all:.1f} s; tokens/s = steps / s / "
                       f"{nl} layers"),
            "one_thread": {"value": d_one / s_one / nl, "cores": 1, "steps": d_one,
                           "seconds": s_one},
            "python_oracle_one_thread": {"value": d_py / s_py / nl, "cores": 1, "steps": d_py,
                                         "seconds": s_py}}


VARIANTS = {}  # mode name -> workload.Variant, filled by main()

# The paper's own headline figures (section 5.3), measured end to end on other
# hardware and software; context only, never a target or a ratio here.
PAPER_CONTEXT = {
    "hardware": "one NVIDIA RTX A6000 (48 GB); FlexGen serving, FlashAttention-2 for dense "
                "attention, a custom Triton kernel for the sparse attention",
    "throughput_vs_dense": {"value": 3.1, "workload": "Lumina-mGPT-7B at its largest feasible "
                            "batch (54 vs 16 for dense); Janus-Pro-7B: 2.3x (batch 96 vs 32)"},
    "latency_vs_dense": {"value": 1.19, "workload": "Lumina-mGPT-7B end to end at 95% sparsity "
                         "(batch 16); Janus-Pro-7B: 1.18x (batch 32)"},
    "attention_only_vs_dense_last_step": {"range": [4.15, 9.78], "workload": "Janus-Pro-7B "
                                          "4.15x / 5.03x at 90% / 95% sparsity, Lumina-mGPT-7B "
                                          "6.52x / 9.78x"},
    "comparable": "no: end-to-end image throughput and latency with model weights on another GPU; "
                  "the paper prints no attention-kernel time, tokens/s or bandwidth",
}


def capture(bt, mode):
    """The whole decode step (every layer) as one HIP graph."""
    import torch
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        run_step(bt, mode)
    return g


def run_step(bt, mode, timers=None):
    from paper_2609_19702_amd import workload
    workload.step(bt, dense=mode == "dense", fused=mode == "fused", timers=timers,
                  variant=VARIANTS.get(mode))


def timed_steps(bt, steps, mode, graph):
    """ms per step over ``steps`` steps (graph replays, or eager launches)."""
    import torch
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record()
    for _ in range(steps):
        if graph is not None:
            graph.replay()
        else:
            run_step(bt, mode)
    end.record()
    torch.cuda.synchronize()
    return start.elapsed_time(end) / steps


def step_distribution(graph, steps):
    """Median, 10th and 90th percentile (ms) of single graph-replayed steps,
    each between its own pair of events; a pass of its own after the timed
    steps, which it does not change."""
    import torch
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(steps)]
    torch.cuda.synchronize()
    for a, b in evs:
        a.record()
        graph.replay()
        b.record()
    torch.cuda.synchronize()
    return percentiles([a.elapsed_time(b) for a, b in evs])


def percentiles(xs):
    q = sorted(xs)

    def at(f):  # linear interpolation between order statistics
        x = f * (len(q) - 1)
        i = int(x)
        return q[i] + (q[min(i + 1, len(q) - 1)] - q[i]) * (x - i)

    return {"median": at(0.5), "p10": at(0.1), "p90": at(0.9), "n": len(q)}


def gpu_clocks():
    """Current shader and memory clocks as rocm-smi reports them (a read-only
    query; None where it is missing or fails)."""
    import shutil
    import subprocess
    exe = shutil.which("rocm-smi")
    if exe is None:
        return None
    try:
        r = subprocess.run([exe, "--showclocks", "--json"], capture_output=True, text=True,
                           timeout=30)
        cards = json.loads(r.stdout)
    except (subprocess.SubprocessError, OSError, ValueError):
        return None
    for card, fields in sorted(cards.items()):
        if isinstance(fields, dict):
            return {"card": card, **{k.rstrip(":"): v for k, v in fields.items() if "clk" in k}}
    return None


def spin_cycles_per_ms():
    """Rate of torch's spin kernel (``torch.cuda._sleep``), measured."""
    import torch
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda._sleep(1000)
    s.record()
    torch.cuda._sleep(1_000_000)
    e.record()
    torch.cuda.synchronize()
    return 1_000_000 / max(s.elapsed_time(e), 1e-3)


def kernel_times(bt, steps, mode, prefill=True):
    """Per-launch duration (ms) of the split-K decode kernel over ``steps``
    eager steps, from events bound to the kernel's own start and end.

    Python issues a layer more slowly than the GPU runs it, so launched one by
    one every kernel would start on an idle GPU.  With ``prefill`` (the
    default) each step is queued behind a spin kernel that lasts twice the
    host's time to issue a step, so the layers then run back to back, as they
    do in the replays of the step's graph.  (Events captured into the graph
    itself do not give usable times here.)"""
    import torch
    from paper_2609_19702_amd import binding as B
    timers = [[B.timing_events() for _ in bt.layers] for _ in range(steps + 1)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    run_step(bt, mode, timers=timers[steps])  # the host's time to issue one step
    host_ms = (time.perf_counter() - t0) * 1e3
    torch.cuda.synchronize()
    prefill = prefill and hasattr(torch.cuda, "_sleep")  # private torch API: time as issued without it
    spin = int(spin_cycles_per_ms() * (2 * host_ms + 0.5)) if prefill else 0
    for k in range(steps):
        if spin:
            torch.cuda._sleep(spin)
        run_step(bt, mode, timers=timers[k])
    torch.cuda.synchronize()
    return [a.elapsed_time(b) for row in timers[:steps] for (a, b) in row]


SWEEP_MIN_BYTES = 1 << 30     # rotating layer buffers per cell: at least 1 GiB of KV ...
SWEEP_MIN_LAYERS = 4          # ... in at least this many layers,
SWEEP_MAX_BYTES = 100 << 30   # ... and at most this much (then at least 2 layers)


def sweep_layers(w):
    """Distinct layer buffers for one sweep cell, so that no launch finds its
    KV in the caches left by the previous one."""
    rows = w.prompt_len + w.decode_len
    lb = w.batch * w.num_kv_heads * rows * w.head_dim * 2 * 2
    n = max(SWEEP_MIN_LAYERS, -(-SWEEP_MIN_BYTES // lb))
    if n * lb > SWEEP_MAX_BYTES:
        n = max(2, SWEEP_MAX_BYTES // lb)
    return n


def run_sweep(args):
    """Per-layer decode time of every Janus-shaped sweep cell in diagonal and
    dense mode: a graph-replayed step over rotating layer buffers (fused
    ``dsa_decode_step`` per layer, or dense ``dsa_decode_attention``), and the
    decode kernel's own duration from events bound to it."""
    import torch
    from paper_2609_19702_amd import binding as B
    from paper_2609_19702_amd import synth, workload
    cells = synth.sweep_workloads()
    if args.cells:
        keys = args.cells.split(",")
        cells = [c for c in cells if any(k in c.name for k in keys)]
    groups = {}
    for c in cells:
        groups.setdefault((c.grid_h, c.batch), []).append(c)
    steps, warm = max(args.steps, 3), max(args.warmup, 1)
    for (g, b), ws in groups.items():
        base = ws[0].with_(name=f"sweep_g{g}_b{b}")
        nl = sweep_layers(base)
        t0 = time.time()
        bt0 = workload.make_batch(base, layers=nl)
        dense_ms = None
        for w in ws:
            bt = workload.with_window(bt0, w.window)
            workload.build_history_shared(bt)
            for mode in ("fused",) + (("dense",) if dense_ms is None else ()):
                for _ in range(warm):
                    run_step(bt, mode)
            torch.cuda.synchronize()
            info, dinfo = B.launch_info(bt.p, bt.s), B.launch_info(bt.pd, bt.s)
            row = {"cell": w.name, "grid": f"{g}x{g}", "batch": b, "window": bt.p.window,
                   "n_att": bt.p.n_att, "no_skip": bt.p.n_att >= bt.p.window,
                   "layers": nl, "positions": "ragged",
                   "launch_threads": info.workgroups * 64 * info.waves_per_group,
                   "dense_launch_threads": dinfo.workgroups * 64 * dinfo.waves_per_group}
            res = {}
            for mode in ("fused",) + (("dense",) if dense_ms is None else ()):
                gr = capture(bt, mode)
                gr.replay()
                torch.cuda.synchronize()
                ms = timed_steps(bt, steps, mode, gr)
                kt = statistics.fmean(kernel_times(bt, steps, mode))
                res[mode] = (ms / nl, kt)
                del gr
            if dense_ms is None:
                dense_ms = res["dense"]
            sp_bytes = bt.kv_bytes(dense=False) / nl
            de_bytes = bt.kv_bytes(dense=True) / nl
            f_ms, f_kt = res["fused"]
            d_ms, d_kt = dense_ms
            row.update({
                "kv_mb_per_layer": sp_bytes / 1e6, "dense_kv_mb_per_layer": de_bytes / 1e6,
                "layer_us": f_ms * 1e3, "decode_kernel_us": f_kt * 1e3,
                "kernel_gbps": sp_bytes / (f_kt * 1e-3) / 1e9,
                "hbm_frac": sp_bytes / (f_kt * 1e-3) / 1e9 / HBM_PEAK_GBPS,
                "dense_layer_us": d_ms * 1e3, "dense_kernel_us": d_kt * 1e3,
                "dense_kernel_gbps": de_bytes / (d_kt * 1e-3) / 1e9,
                "speedup_vs_dense": d_ms / f_ms, "ideal_speedup": de_bytes / sp_bytes,
                "tokens_per_s_per_layer": b / (f_ms * 1e-3),
            })
            print(json.dumps(row), flush=True)
            del bt
        print(f"# {base.name}: {nl} layers, {time.time() - t0:.1f}s", file=sys.stderr, flush=True)
        del bt0
        torch.cuda.empty_cache()


def run_trajectory(args):
    """One whole image per request: decode positions 0 .. H*W-1 in order, every
    layer per position, starting from empty selection states, so phase 1, the
    phase-2 selections and phase 3 all occur as often as they do in
    generation.  Each position's step (all layers) is captured as one HIP
    graph reading its positions from a device table; the graphs are replayed
    back to back and timed with events, for the fused step and for dense
    mode.  The K/V rows of every position are in the cache from the start
    (the model would write row t just before step t)."""
    import torch
    from paper_2609_19702_amd import binding as B
    from paper_2609_19702_amd import synth, workload
    w = synth.WORKLOADS[args.workload].with_(positions="last")
    if args.batch:
        w = w.with_(batch=args.batch, name=f"{w.name}_b{args.batch}")
    t0 = time.time()
    bt = workload.make_batch(w)
    L_dec = w.decode_len
    table = torch.arange(L_dec, dtype=torch.int32, device="cuda").repeat_interleave(w.batch)
    table = table.view(L_dec, w.batch)
    res = {"metric": "whole-image decode attention time (all positions, all layers)",
           "workload": f"{w.name}_like", "layers": len(bt.layers), "batch": w.batch,
           "positions": L_dec, "window": bt.p.window, "n_att": bt.p.n_att,
           "launch": "hip_graph per position",
           "kept_lists": B.launch_info(bt.p, bt.s).kept_read}
    for mode in ("fused", "dense"):
        for L in bt.layers:
            B.state_reset(bt.p, bt.s, L.bufs.state)
        graphs = []
        for t in range(L_dec):
            bt.pos = table[t]
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                run_step(bt, mode)
            graphs.append(g)
        torch.cuda.synchronize()
        for L in bt.layers:  # capture ran nothing; start the trajectory from empty states
            B.state_reset(bt.p, bt.s, L.bufs.state)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for g in graphs:
            g.replay()
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1)
        res[mode] = {"ms": ms, "us_per_position": ms * 1e3 / L_dec,
                     "tokens_per_s": w.batch * L_dec / (ms * 1e-3)}
        if mode == "fused":
            cnt, flg, _ = B.state_views(bt.p, bt.s, bt.layers[0].bufs.state)
            res["fused"]["skip_entries_per_head"] = int(cnt.max().item())
            res["fused"]["skip_capacity"] = B.state_layout(bt.p, bt.s).cap
            res["fused"]["state_flags"] = int(flg.any().item())
        del graphs
        print(f"# {mode}: {ms:.1f} ms ({time.time() - t0:.1f}s)", file=sys.stderr, flush=True)
    res["speedup_vs_dense"] = res["dense"]["ms"] / res["fused"]["ms"]
    print(json.dumps(res), flush=True)


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}); the decode path has no "
              "cross-GPU step: requests and heads shard with no exchange", file=sys.stderr)
        sys.exit(2)
    import torch
    from paper_2609_19702_amd import synth, workload
    from paper_2609_19702_amd import binding as B
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    B.lib()
    if args.calibrate_copy:
        n = args.calibrate_copy << 20
        src = torch.ones(n, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(10):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"calibrate_copy_bytes": n, "launches": 10}))
        return
    if args.sweep:
        run_sweep(args)
        return
    if args.trajectory:
        run_trajectory(args)
        return
    w = synth.WORKLOADS[args.workload]
    if args.positions:
        w = w.with_(positions=args.positions)
    t0 = time.time()
    bt = workload.make_batch(w)
    workload.build_histories(bt)
    modes = (args.only,) if args.only else ("fused", "separate", "dense", "diag_sink4", "streaming",
                                             "fp8_kv", "ring")
    if "diag_sink4" in modes:
        VARIANTS["diag_sink4"] = workload.make_variant(bt, "diag_sink4", B.MODE_DIAGONAL, 4)
    if "streaming" in modes:
        VARIANTS["streaming"] = workload.make_variant(bt, "streaming", B.MODE_WINDOW, 4)
    if "fp8_kv" in modes:
        VARIANTS["fp8_kv"] = workload.make_variant(bt, "fp8_kv", B.MODE_DIAGONAL, 0, fp8=True)
    if "ring" in modes:
        VARIANTS["ring"] = workload.make_ring_variant(bt)
    torch.cuda.synchronize()
    print(f"# setup {time.time() - t0:.1f}s: {w.name} layers={len(bt.layers)} batch={w.batch} "
          f"n_att={bt.p.n_att} window={bt.p.window}", file=sys.stderr, flush=True)

    for _ in range(args.warmup):
        for mode in modes:
            run_step(bt, mode)
    torch.cuda.synchronize()
    graphs = {m: (None if args.eager else capture(bt, m)) for m in modes}
    for g in graphs.values():
        if g is not None:
            g.replay()
    torch.cuda.synchronize()
    ms = {m: timed_steps(bt, args.steps, m, graphs[m]) for m in modes}
    launch = {m: kernel_times(bt, args.steps, m, prefill=not args.eager) for m in modes}
    dist = None
    if graphs.get("fused") is not None:
        dist = step_distribution(graphs["fused"], args.steps)
    if args.only:
        print(json.dumps({"only": args.only, "ms_per_step": ms[args.only],
                          "decode_launch_us": statistics.fmean(launch[args.only]) * 1e3}))
        return
    ms_sparse, ms_dense = ms["fused"], ms["dense"]
    launch_sparse, launch_dense = launch["fused"], launch["dense"]
    print(f"# ms/step ({'eager' if args.eager else 'graph'}): "
          + ", ".join(f"{m} {ms[m]:.3f}" for m in modes)
          + "; decode kernel us: " + ", ".join(f"{m} {statistics.fmean(launch[m]) * 1e3:.2f}" for m in modes),
          file=sys.stderr, flush=True)

    n_layers = len(bt.layers)
    bytes_sparse = bt.kv_bytes(dense=False)
    bytes_dense = bt.kv_bytes(dense=True)
    per_launch = bytes_sparse / n_layers
    mean_launch_ms = statistics.fmean(launch_sparse)
    achieved = per_launch / (mean_launch_ms * 1e-3) / 1e9
    dense_launch_ms = statistics.fmean(launch_dense)
    info = B.launch_info(bt.p, bt.s)
    src_hash = kernel_source_hash()
    traffic = traffic_for(w.name, src_hash)

    base = None
    if not args.no_cpu_baseline:
        base = cpu_baseline(bt, args.cpu_seconds)

    res = {
        "metric": METRIC,
        "value": w.batch / (ms_sparse * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_sparse,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": f"{w.name}_like", "layers": n_layers, "batch": w.batch,
            "q_heads": w.num_q_heads, "kv_heads": w.num_kv_heads, "head_dim": w.head_dim,
            "prompt_len": w.prompt_len, "grid": f"{w.grid_h}x{w.grid_w}", "window": bt.p.window,
            "n_att": bt.p.n_att, "sparsity": round(1 - bt.p.n_att / w.decode_len, 4),
            "positions": w.positions, "accumulate": "fp32",
            "splits": info.max_splits, "rows_per_split": info.rows_per_split,
            "launch": "eager" if args.eager else "hip_graph",
        },
        "kv_gbps": bytes_sparse / (ms_sparse * 1e-3) / 1e9,
        "kv_hbm_frac": bytes_sparse / (ms_sparse * 1e-3) / 1e9 / HBM_PEAK_GBPS,
        "dense": {
            "ms_per_step": ms_dense, "tokens_per_s": w.batch / (ms_dense * 1e-3),
            "kv_gbps": bytes_dense / (ms_dense * 1e-3) / 1e9,
            "decode_launch_us": dense_launch_ms * 1e3,
            "decode_launch_gbps": bytes_dense / n_layers / (dense_launch_ms * 1e-3) / 1e9,
        },
        "separate_calls": {
            "ms_per_step": ms["separate"], "tokens_per_s": w.batch / (ms["separate"] * 1e-3),
            "decode_launch_us": statistics.fmean(launch["separate"]) * 1e3,
        },
        "variants": {
            m: {"ms_per_step": ms[m], "tokens_per_s": w.batch / (ms[m] * 1e-3),
                "decode_launch_us": statistics.fmean(launch[m]) * 1e3,
                "decode_launch_gbps": bt.kv_bytes(False, 1 if m == "fp8_kv" else 2) / n_layers
                / (statistics.fmean(launch[m]) * 1e-3) / 1e9,
                "mode": {"diag_sink4": "diagonal, 4 sinks", "streaming": "window, 4 sinks",
                         "fp8_kv": "diagonal, fp8 E4M3 KV with per-(request, KV head) scales",
                         "ring": "diagonal, ring cache of R = N_r decode slots (physical "
                                 "eviction)"}[m]}
            for m in ("diag_sink4", "streaming", "fp8_kv", "ring")
        },
        "speedup_vs_dense": ms_dense / ms_sparse,
        "ideal_speedup": bytes_dense / bytes_sparse,
        "roofline": {
            "bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
            "frac": achieved / HBM_PEAK_GBPS, "traffic": traffic,
            "kernel": ((("decode_mfma_kernel" if info.kernel_variant == 100 else "decode_kernel")
                        + (" + combine_select_kernel (fused step, one interval)"
                           if info.max_splits > 1 else " (fused step)"))),
            "bytes_per_launch": per_launch,
            "launches_timed": len(launch_sparse),
            "launch_timing": "eager" if args.eager else "eager_back_to_back",
            # every kernel of one layer in the timed replays, launch gaps included
            "layer_us_in_step": ms_sparse * 1e3 / n_layers,
            "launch_us": mean_launch_ms * 1e3, "source_hash": src_hash,
            "launch_us_dist": {k: (v * 1e3 if k != "n" else v)
                               for k, v in percentiles(launch_sparse).items()},
        },
        # single graph-replayed steps, timed apart from the steps above
        "step_ms_dist": dist,
        # read once the timed work is over (a query during it would perturb it)
        "gpu_clocks_after_run": gpu_clocks(),
        "cpu_baseline": base,
        "paper_context": PAPER_CONTEXT,
    }
    if "ring" in VARIANTS:
        ring = VARIANTS["ring"]
        R = ring.ring_rows
        row_bytes = w.num_kv_heads * w.head_dim * 2 * 2 * w.batch  # K and V, bf16, all requests
        res["variants"]["ring"].update({
            "ring_rows": R,
            "kv_resident_bytes_per_layer": (w.prompt_len + R) * row_bytes,
            "linear_kv_resident_bytes_per_layer": (w.prompt_len + w.decode_len) * row_bytes,
            "step_vs_linear": ms["ring"] / ms_sparse,
            "outputs_match_linear": all(torch.equal(L.bufs.out, bf.out)
                                        for L, bf in zip(bt.layers, ring.bufs)),
        })
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
