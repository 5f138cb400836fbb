#!/usr/bin/env python3
"""Benchmark of the SLA hot path on one MI355X.

Default workload: the training step on Waymo-like frame shapes -- segment build
(window-id sort, offsets, chunk plan) + SLA forward + SLA backward, fp16 storage
with fp32 accumulation, H = 4 heads of d = 32 (C = 128), ~60k voxels in 1,521
window slots, rows re-shuffled every step so the builder really sorts.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--config 5]

Prints ONE JSON line.  `value` is voxels per second over the timed K steps
(inputs resident in HBM, buffers rotated over enough sets that the 256 MB
Infinity Cache cannot serve repeats).  The timed steps are replayed from HIP
graphs, one per buffer set, so host launch overhead is not measured.  A second,
eager pass times every phase with HIP events on the launch stream
(`breakdown_ms`, launch gaps included).  The dominant kernel's average duration,
which gives `roofline.achieved`, comes from a graph of back-to-back launches of
that kernel alone over the rotating buffer sets.  `cpu_baseline`
times the CPU oracle (test infrastructure) on a bounded sample on this host.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0       # MI355X HBM3E, AMD published peak
MALL_BYTES = 256 << 20      # Infinity Cache
METRIC = "SLA fwd+bwd voxels/s and ms/frame (N≈60k, C=128); % of HBM roofline"


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=300)
    p.add_argument("--warmup", type=int, default=30)
    p.add_argument("--config", type=int, default=5, choices=[1, 2, 3, 4, 5])
    p.add_argument("--chunk-rows", type=int, default=0)
    p.add_argument("--no-graph", action="store_true", help="time eager launches instead of graph replay")
    p.add_argument("--feature-map", choices=["elu1", "relu"], default=None,
                   help="time the sla_forward_ex / sla_backward_ex variant with this feature map")
    p.add_argument("--eps", type=float, default=None, help="epsilon of the normaliser (with --feature-map)")
    p.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    p.add_argument("--cpu-seconds", type=float, default=12.0)
    p.add_argument("--copy-probe", action="store_true",
                   help="after timing, run plain copies of known size (calibrates PMC byte counters)")
    p.add_argument("--projected", action="store_true",
                   help="time the projection fused into SLA (sla_forward_projected) against the unfused "
                        "chain: torch linear, sla_forward, torch linear")
    p.add_argument("--cwi", action="store_true",
                   help="time the cross-window interaction (cell table build + forward) on a Waymo-like "
                        "pillar frame")
    p.add_argument("--xca", action="store_true",
                   help="time the XCA variant (sla_forward_xca) beside sla_forward on one frame, plan "
                        "built outside the timed region")
    p.add_argument("--compare-scatter", action="store_true",
                   help="instead of the training step: forward time and memory of the chunk-wise path "
                        "against the naive scatter-based one, as sequence length and window length grow")
    p.add_argument("--pmc-summary", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                   help="no GPU work: summarise two rocprofv3 --pmc counter_collection.csv files "
                        "(FETCH_SIZE run, WRITE_SIZE run) of `bench.py --no-graph --copy-probe`")
    p.add_argument("--sq-summary", nargs="+", metavar="CSV",
                   help="no GPU work: summarise rocprofv3 --pmc counter_collection.csv files of SQ "
                        "counters (`bench.py --no-graph` runs): MFMA and VALU busy, LDS bank conflicts")
    return p.parse_args()


def elem_size(dtype):
    return {"f32": 4, "f16": 2, "bf16": 2}[dtype]


COPY_PROBE_BYTES = 256 << 20   # per copy, 3 copies from distinct buffers
KERNEL_SOURCES = ["paper_2401_00912_amd/csrc/sla_attn.hip", "paper_2401_00912_amd/csrc/sla_attn_core.h",
                  "paper_2401_00912_amd/csrc/sla_common.h"]
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "k_sla_bwd_training_step_pmc.txt")


def kernel_source_hash():
    import hashlib

    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def short_kernel(name):
    for k in ("k_sla_bwd", "k_sla_fwd_proj", "k_sla_fwd", "k_sort", "k_merge", "k_plan", "k_cwi_tiled",
              "k_cwi_fwd", "k_cwi_dw_reduce", "k_cwi_dw", "k_cwi_map", "k_cwi_clear", "k_xca_fwd_mma",
              "k_xca_bwd_mma", "k_xca_fwd", "k_xca_bwd", "k_xca_dtau", "k_out_proj", "k_rows_gemm",
              "k_wgrad_reduce", "k_wgrad", "k_prep"):
        if k in name:
            return k
    if "copyBuffer" in name:    # the runtime's device-to-device copy kernel
        return "copy"
    return None


def pmc_summary(fetch_csv, write_csv):
    """Per-dispatch FETCH_SIZE / WRITE_SIZE of every kernel of the step, scaled by
    what the same counters read for the plain copy of known size."""
    import csv

    def per_kernel(path, counter):
        acc = {}
        with open(path) as fh:
            for r in csv.DictReader(fh):
                if r["Counter_Name"] != counter:
                    continue
                k = short_kernel(r["Kernel_Name"])
                if k is None:
                    continue
                acc.setdefault(k, []).append(float(r["Counter_Value"]) * 1024.0)  # KiB -> bytes
        if "copy" in acc:          # the probe's copies, not the binding's small ones
            acc["copy"] = [x for x in acc["copy"] if x > 0.01 * COPY_PROBE_BYTES] or acc.pop("copy")
        return {k: (float(np.mean(v)), len(v)) for k, v in acc.items() if v}

    f, w = per_kernel(fetch_csv, "FETCH_SIZE"), per_kernel(write_csv, "WRITE_SIZE")
    if "copy" not in f or "copy" not in w:
        raise SystemExit("pmc summary: no copy-probe dispatch in the counter files")
    ff, fw = f["copy"][0] / COPY_PROBE_BYTES, w["copy"][0] / COPY_PROBE_BYTES
    lines = [
        f"kernel_source_sha256: {kernel_source_hash()}",
        f"copy_probe_bytes: {COPY_PROBE_BYTES}",
        f"fetch_factor: {ff:.4f}   (FETCH_SIZE bytes read by the copy / bytes it reads)",
        f"write_factor: {fw:.4f}   (WRITE_SIZE bytes by the copy / bytes it writes)",
        "kernel      dispatches  FETCH_raw_B   WRITE_raw_B   fetch_scaled_B  write_scaled_B  traffic_scaled_B",
    ]
    for k in ("k_sort", "k_merge", "k_plan", "k_sla_fwd", "k_sla_bwd", "k_cwi_clear", "k_cwi_map",
              "k_cwi_tiled", "k_cwi_fwd", "k_cwi_dw", "k_cwi_dw_reduce", "copy"):
        if k in f and k in w:
            fr, wr = f[k][0], w[k][0]
            lines.append(f"{k:<11} {f[k][1]:>10}  {fr:>12.0f}  {wr:>12.0f}  {fr / ff:>14.0f}  "
                         f"{wr / fw:>14.0f}  {fr / ff + wr / fw:>16.0f}")
    return "\n".join(lines)


MI355X_CUS, MI355X_SIMDS, MI355X_XCDS = 256, 1024, 8


def sq_summary(paths):
    """Per-launch SQ counters of every kernel of the step (mean over dispatches)
    and the derived figures rocprofv3 defines for gfx950: MfmaUtil = MFMA-busy
    cycles / (GPU-active cycles x SIMDs), VALUBusy = VALU-active cycles / CUs /
    GPU-active cycles, LDS bank-conflict ratio = conflict cycles / (LDS-active -
    conflict cycles), and LDS-active cycles per CU over GPU-active cycles.  The counter file sums GRBM_GUI_ACTIVE over the 8 XCDs
    while those definitions take its per-XCD maximum, so the sum is divided by 8.
    One F16 MFMA "MOP" is 512 flops; TFLOP/s is over the dispatch's own duration
    (its start and end timestamps)."""
    import csv

    acc, dur = {}, {}
    for path in paths:
        seen = set()
        with open(path) as fh:
            for r in csv.DictReader(fh):
                k = short_kernel(r["Kernel_Name"])
                if k is None or k == "copy":
                    continue
                acc.setdefault(k, {}).setdefault(r["Counter_Name"], []).append(float(r["Counter_Value"]))
                if r["Dispatch_Id"] not in seen:
                    seen.add(r["Dispatch_Id"])
                    dur.setdefault(k, []).append((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-9)
    lines = ["kernel      counter                          per_launch        dispatches"]
    step = ("k_sort", "k_merge", "k_sla_fwd", "k_sla_bwd")
    for k in [x for x in step if x in acc] + sorted(set(acc) - set(step)):
        c = {name: float(np.mean(v)) for name, v in acc[k].items()}
        for name in sorted(c):
            lines.append(f"{k:<11} {name:<32} {c[name]:>16.0f}  {len(acc[k][name]):>10}")
        t = float(np.median(dur[k]))
        lines.append(f"{k:<11} derived dispatch_us_median        {t * 1e6:>16.2f}")
        g = c.get("GRBM_GUI_ACTIVE")
        if g:
            g /= MI355X_XCDS
            if "SQ_VALU_MFMA_BUSY_CYCLES" in c:
                lines.append(f"{k:<11} derived MfmaUtil_percent          "
                             f"{100 * c['SQ_VALU_MFMA_BUSY_CYCLES'] / (g * MI355X_SIMDS):>16.2f}")
            if "SQ_ACTIVE_INST_VALU" in c:
                lines.append(f"{k:<11} derived VALUBusy_percent          "
                             f"{100 * c['SQ_ACTIVE_INST_VALU'] / MI355X_CUS / g:>16.2f}")
            if "SQ_LDS_IDX_ACTIVE" in c:   # as VALUBusy: LDS-active cycles per CU over GPU-active cycles
                lines.append(f"{k:<11} derived LdsActive_percent         "
                             f"{100 * c['SQ_LDS_IDX_ACTIVE'] / MI355X_CUS / g:>16.2f}")
        if "SQ_LDS_BANK_CONFLICT" in c and "SQ_LDS_IDX_ACTIVE" in c:
            den = c["SQ_LDS_IDX_ACTIVE"] - c["SQ_LDS_BANK_CONFLICT"]
            if den > 0:
                lines.append(f"{k:<11} derived LdsBankConflict_ratio     {c['SQ_LDS_BANK_CONFLICT'] / den:>16.4f}")
        if "SQ_INSTS_VALU_MFMA_MOPS_F16" in c:
            fl = 512 * c["SQ_INSTS_VALU_MFMA_MOPS_F16"]
            lines.append(f"{k:<11} derived MFMA_F16_flops            {fl:>16.0f}")
            lines.append(f"{k:<11} derived MFMA_F16_TFLOPs           {fl / t / 1e12:>16.1f}")
    return "\n".join(lines)


def stored_traffic(kernel):
    """Scaled HBM bytes per launch of `kernel` from the committed counter summary,
    or None when there is none or the kernel source changed since it was taken."""
    try:
        with open(TRAFFIC_FILE) as fh:
            text = fh.read().splitlines()
    except OSError:
        return None
    sha = next((l.split()[1] for l in text if l.startswith("kernel_source_sha256:")), None)
    if sha != kernel_source_hash():
        return None
    for l in text:
        parts = l.split()
        if parts and parts[0] == kernel and len(parts) == 7:
            return float(parts[6])
    return None


def time_rotating(torch, dev, fn, sets, reps, warmup, eager=False):
    """Average microseconds of one call of fn over the buffer sets in rotation:
    one HIP graph holding one call per set, replayed under events on the current
    stream (a graph per call would time the host's graph launches for short calls),
    or eager launches."""
    nsets = len(sets)
    for i in range(warmup):
        fn(sets[i % nsets])
    torch.cuda.synchronize()
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    if eager:
        t0.record()
        for i in range(reps):
            fn(sets[i % nsets])
        t1.record()
        torch.cuda.synchronize()
        return t0.elapsed_time(t1) / reps * 1e3
    cur = torch.cuda.current_stream(dev)
    cap = torch.cuda.Stream(dev)
    cap.wait_stream(cur)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(cap):
        with torch.cuda.graph(g, stream=cap):
            for st in sets:
                fn(st)
    cur.wait_stream(cap)
    g.replay()
    torch.cuda.synchronize()
    rounds = max(1, reps // nsets)
    t0.record()
    for _ in range(rounds):
        g.replay()
    t1.record()
    torch.cuda.synchronize()
    return t0.elapsed_time(t1) / (rounds * nsets) * 1e3


def main():
    args = parse()
    if args.pmc_summary:
        print(pmc_summary(*args.pmc_summary))
        return
    if args.sq_summary:
        print(sq_summary(args.sq_summary))
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {args.gpus}); "
              "SLA would shard by contiguous window ranges with no exchange between GPUs", file=sys.stderr)
        sys.exit(2)
    import torch

    import workloads
    from paper_2401_00912_amd import sla

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    sla.lib()
    if args.compare_scatter:
        print(json.dumps(compare_scatter(torch, sla, workloads, dev)), flush=True)
        return
    if args.cwi:
        print(json.dumps(bench_cwi(torch, sla, workloads, dev, args)), flush=True)
        return
    if args.projected:
        print(json.dumps(bench_projected(torch, sla, workloads, dev, args)), flush=True)
        return
    if args.xca:
        print(json.dumps(bench_xca(torch, sla, workloads, dev, args)), flush=True)
        return

    cfg = args.config
    training = cfg == 5
    variant = None
    if args.feature_map is not None or args.eps is not None:
        variant = (args.feature_map or "elu1", 0.0 if args.eps is None else args.eps)
    base = workloads.make_config(cfg, with_grad=training)
    n, H, d, W, dt = base["n"], base["heads"], base["head_dim"], base["num_windows"], base["dtype"]
    e = elem_size(dt)
    C = H * d
    row_bytes = C * e
    tdt = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}[dt]

    def dev_vals(a):
        t = torch.from_numpy(np.ascontiguousarray(a))
        if dt == "bf16":
            t = t.view(torch.bfloat16)
        return t.to(dev)

    per_set = (8 if training else 4) * n * row_bytes + 8 * n + sla.plan_bytes(n, W)
    nsets = max(3, int(np.ceil(2 * MALL_BYTES / per_set)) + 1)
    sets = []
    for s in range(nsets):
        wl = workloads.shuffled(base, [cfg, 2, s]) if base["ids"] is not None else base
        st = {
            "q": dev_vals(wl["q"]), "k": dev_vals(wl["k"]), "v": dev_vals(wl["v"]),
            "o": torch.empty((n, H, d), dtype=tdt, device=dev),
        }
        if base["ids"] is not None:
            st["ids"] = torch.from_numpy(wl["ids"]).to(dev)
        else:
            st["offsets"] = torch.from_numpy(wl["offsets"].astype(np.int32)).to(dev)
        st["plan_buf"] = sla.new_plan_buffer(n, W, dev)
        if training:
            st["dout"] = dev_vals(wl["dout"])
            st["dq"] = torch.empty_like(st["q"])
            st["dk"] = torch.empty_like(st["q"])
            st["dv"] = torch.empty_like(st["q"])
        sets.append(st)

    def build(st):
        if "ids" in st:
            return sla.build_segments(st["ids"], num_windows=W, chunk_rows=args.chunk_rows,
                                      plan_buf=st["plan_buf"], want_perm=False)
        return sla.build_segments(None, num_windows=W, chunk_rows=args.chunk_rows, offsets=st["offsets"],
                                  n=n, plan_buf=st["plan_buf"])

    plans = [build(st) for st in sets]   # forward-only configs time forward given a plan
    torch.cuda.synchronize()

    def step(i, ev=None):
        st = sets[i % nsets]
        if ev is not None:
            ev[0].record()
        if training:
            plan = build(st)
        else:
            plan = plans[i % nsets]
        if ev is not None:
            ev[1].record()
        sla.forward(plan, st["q"], st["k"], st["v"], out=st["o"], feature_map=args.feature_map, eps=args.eps)
        if ev is not None:
            ev[2].record()
        if training:
            sla.backward(plan, st["q"], st["k"], st["v"], st["dout"], st["dq"], st["dk"], st["dv"],
                         feature_map=args.feature_map, eps=args.eps)
        if ev is not None:
            ev[3].record()

    stream = torch.cuda.current_stream(dev)
    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()

    # ---- headline: K steps, graph replay (one graph per buffer set)
    graphs = None
    if not args.no_graph:
        try:
            graphs = []
            cap = torch.cuda.Stream(dev)
            cap.wait_stream(stream)
            with torch.cuda.stream(cap):
                for s in range(nsets):
                    g = torch.cuda.CUDAGraph()
                    with torch.cuda.graph(g, stream=cap):
                        step(s)
                    graphs.append(g)
            stream.wait_stream(cap)
            for g in graphs:          # replays must reproduce eager results: run each once
                g.replay()
            torch.cuda.synchronize()
        except Exception as exc:  # noqa: BLE001
            print(f"bench.py: graph capture unavailable ({exc}); timing eager launches", file=sys.stderr)
            graphs = None
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0.record()
    for i in range(args.steps):
        if graphs is not None:
            graphs[i % nsets].replay()
        else:
            step(i)
    t1.record()
    torch.cuda.synchronize()
    ms_total = t0.elapsed_time(t1)
    ms_step = ms_total / args.steps
    # four more loops of K steps, for the median of five (the first loop is `value`)
    loops = [ms_step]
    for _ in range(4):
        t0.record()
        for i in range(args.steps):
            if graphs is not None:
                graphs[i % nsets].replay()
            else:
                step(i)
        t1.record()
        torch.cuda.synchronize()
        loops.append(t0.elapsed_time(t1) / args.steps)
    e2e_ms = None
    if not training:
        # forward-only configs: end to end, segment build + forward, eager launches
        for i in range(args.warmup):
            sla.forward(build(sets[i % nsets]), sets[i % nsets]["q"], sets[i % nsets]["k"],
                        sets[i % nsets]["v"], out=sets[i % nsets]["o"])
        torch.cuda.synchronize()
        t0.record()
        for i in range(args.steps):
            st = sets[i % nsets]
            sla.forward(build(st), st["q"], st["k"], st["v"], out=st["o"])
        t1.record()
        torch.cuda.synchronize()
        e2e_ms = t0.elapsed_time(t1) / args.steps

    # ---- per-kernel breakdown: eager launches bracketed by events on the launch stream.
    # A spin kernel first lets the host enqueue every step before the GPU reaches them,
    # so the events bracket device time only.
    nb = min(args.steps, 100)
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(nb)]
    torch.cuda.synchronize()
    try:
        torch.cuda._sleep(int(2e8))
    except Exception:  # noqa: BLE001
        pass
    for i in range(nb):
        step(i, evs[i])
    torch.cuda.synchronize()
    t_build = float(np.mean([a[0].elapsed_time(a[1]) for a in evs])) if training else 0.0
    t_fwd = float(np.mean([a[1].elapsed_time(a[2]) for a in evs]))
    t_bwd = float(np.mean([a[2].elapsed_time(a[3]) for a in evs])) if training else 0.0

    fwd_bytes = 4 * n * row_bytes
    bwd_bytes = 7 * n * row_bytes
    if training:
        dom, dom_ms_eager, dom_bytes = "k_sla_bwd", t_bwd, bwd_bytes
    else:
        dom, dom_ms_eager, dom_bytes = "k_sla_fwd", t_fwd, fwd_bytes

    # ---- the dominant kernel alone: one graph of back-to-back launches over the
    # rotating buffer sets (each set's plan as the steps built it), replayed under
    # events on the launch stream.  Nodes of one graph start closer together than
    # eager launches, so this is nearer the kernel's own duration.
    dom_ms = dom_ms_eager
    dom_launches = 0
    if graphs is not None:
        def dom_call(s_):
            st = sets[s_ % nsets]
            if training:
                sla.backward(plans[s_ % nsets], st["q"], st["k"], st["v"], st["dout"], st["dq"], st["dk"],
                             st["dv"], feature_map=args.feature_map, eps=args.eps)
            else:
                sla.forward(plans[s_ % nsets], st["q"], st["k"], st["v"], out=st["o"],
                            feature_map=args.feature_map, eps=args.eps)
        per_graph = 2 * nsets
        gd = torch.cuda.CUDAGraph()
        cap = torch.cuda.Stream(dev)
        cap.wait_stream(stream)
        with torch.cuda.stream(cap):
            with torch.cuda.graph(gd, stream=cap):
                for s_ in range(per_graph):
                    dom_call(s_)
        stream.wait_stream(cap)
        gd.replay()
        torch.cuda.synchronize()
        reps = max(5, args.steps // per_graph)
        t0.record()
        for _ in range(reps):
            gd.replay()
        t1.record()
        torch.cuda.synchronize()
        dom_launches = reps * per_graph
        dom_ms = t0.elapsed_time(t1) / dom_launches
        del gd
    achieved = dom_bytes / (dom_ms * 1e-3) / 1e9

    if args.copy_probe:
        copy_probe(torch, dev)
    step_bytes = (fwd_bytes + bwd_bytes + 8 * n) if training else fwd_bytes
    copy_gbs = measure_copy(torch, dev)
    perms = None
    if "ids" in sets[0]:   # the plans' permutations (rows arrive unsorted)
        lay = sla.plan_layout(n, W)
        perms = [p.buf[lay.perm: lay.perm + 4 * n].view(torch.int32) for p in plans]
    gather_gbs = measure_gather(torch, dev, sets, perms, ("q", "k", "v", "dout") if training else ("q", "k", "v"))

    nonempty = int((np.diff(plans[0].offsets.cpu().numpy()) > 0).sum())
    frames = base.get("frames", 1)
    out = {
        "metric": METRIC,
        "value": n / (ms_step * 1e-3),
        "unit": "voxels/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "ms_per_frame": ms_step / frames,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": dt,
        "data": "synthetic",
        "config": {
            "workload": base["name"],
            "phases": "build+forward+backward" if training else "forward (plan built outside the timed region)",
            "n": n, "heads": H, "head_dim": d, "num_windows": W, "nonempty_windows": nonempty,
            "frames": frames, "buffer_sets": nsets, "graph_replay": graphs is not None,
            "chunk_rows": args.chunk_rows or int(sla.lib().sla_default_chunk_rows()),
        },
        "roofline": {
            "bound": "hbm",
            "kernel": dom,
            "achieved": achieved,
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": achieved / HBM_PEAK_GBS,
            # the stored counters were taken for the default feature map
            "traffic": stored_traffic(dom) if variant is None else None,
            "algorithmic_bytes": dom_bytes,
            "avg_ms": dom_ms,
            # how avg_ms was taken: a graph of back-to-back launches of the kernel
            # (launches counted), or the eager breakdown's events (launch gaps included)
            "avg_ms_launches": dom_launches,
            "avg_ms_eager": dom_ms_eager,
            # a plain device-to-device copy on the same GPU, for scale
            "copy_gbs": copy_gbs,
            "frac_of_copy": achieved / copy_gbs if copy_gbs else None,
            # torch's index_select of the kernel's input rows through the same
            # permutation (gathered reads, contiguous writes), for scale
            "gather_gbs": gather_gbs,
            "frac_of_gather": achieved / gather_gbs if gather_gbs else None,
        },
        "breakdown_ms": {"build": t_build, "forward": t_fwd, "backward": t_bwd},
        "step_roofline_frac": step_bytes / (ms_step * 1e-3) / 1e9 / HBM_PEAK_GBS,
        "ms_per_step_loops": loops,
        "ms_per_step_median_of_5": float(np.median(loops)),
    }
    if e2e_ms is not None:
        out["build_plus_forward_ms"] = e2e_ms
    if variant is not None:
        out["config"]["feature_map"], out["config"]["eps"] = variant
    if not args.no_cpu:
        out["cpu_baseline"] = cpu_baseline(base, training, args.cpu_seconds, variant)
        out["cpu_baseline"]["all_cores"] = cpu_baseline_pool(cfg, training, args.cpu_seconds, variant)
    print(json.dumps(out), flush=True)


def bench_cwi(torch, sla, workloads, dev, args):
    """Cross-window interaction on Waymo-like pillar frames (C = 128, 13-tap axis
    kernels, fp16): the cell table build and the forward, rows visited in the
    window order of the frame's SLA plan (and, for comparison, in row order);
    buffer sets rotated, graph replay."""
    nsets = 6
    sets = []
    for s_ in range(nsets):
        f = workloads.make_cwi_frame(seed=s_)
        # the window order comes from the library's own plan of the frame
        plan = sla.build_segments(torch.from_numpy(f["ids"].astype(np.int32)).to(dev), f["num_windows"])
        dt = {"f16": torch.float16}[f["dtype"]]
        sets.append({
            "coords": torch.from_numpy(f["coords"]).to(dev),
            "order": plan.perm,
            "x": torch.from_numpy(f["x"]).to(dev),
            "w": [torch.from_numpy(f[k]).to(dev) for k in ("w_x", "w_y", "w_3")],
            "y": torch.empty(f["n"], f["channels"], dtype=dt, device=dev),
            "dy": torch.from_numpy(workloads.cast_values(
                np.random.default_rng([7, s_]).standard_normal(f["x"].shape).astype(np.float32),
                f["dtype"])).to(dev),
            "dx": torch.empty(f["n"], f["channels"], dtype=dt, device=dev),
            "dw": [torch.empty(f[k].shape, dtype=dt, device=dev) for k in ("w_x", "w_y", "w_3")],
            "ws": torch.empty(sla.cwi_backward_workspace_bytes(f["n"], dt, f["channels"], f["w_x"].shape[0],
                                                               f["w_y"].shape[0]),
                              dtype=torch.uint8, device=dev),
            "map": torch.empty(sla.cwi_map_bytes(*f["grid"]) // 4, dtype=torch.int32, device=dev),
            "grid": f["grid"], "n": f["n"], "C": f["channels"],
        })

    def build(st):
        sla.cwi_build_map(st["coords"], st["grid"], map=st["map"])

    def fwd(st, ordered=True):
        sla.cwi_forward(st["map"], st["grid"], st["coords"], st["x"], *st["w"],
                        order=st["order"] if ordered else None, y=st["y"])

    def bwd(st):
        sla.cwi_backward(st["map"], st["grid"], st["coords"], st["x"], *st["w"], st["dy"], order=st["order"],
                         workspace=st["ws"], out=(st["dx"], *st["dw"]))

    def timed(fn, reps):
        return time_rotating(torch, dev, fn, sets, reps, args.warmup, eager=args.no_graph)

    reps = max(100, args.steps) if not args.no_graph else args.steps
    for st in sets:
        build(st)
    t_build = timed(build, reps)
    t_fwd = timed(fwd, reps)
    t_fwd_rows = timed(lambda st: fwd(st, ordered=False), reps)
    t_bwd = timed(bwd, reps)
    n = int(np.mean([st["n"] for st in sets]))
    C, e = sets[0]["C"], 2
    cells = int(np.prod(sets[0]["grid"]))
    fwd_bytes = n * (2 * C * e + 12 + 4)          # x read, y written, coordinates, visiting order
    # backward: dy read and dx written (the reversed-kernel pass), then x and dy
    # of the three convolution quarters read again for the kernel gradients,
    # coordinates and visiting order read by both passes
    bwd_bytes = n * (2 * C * e + 2 * (3 * C // 4) * e + 2 * (12 + 4))
    build_bytes = 4 * cells + n * (12 + 4)        # table cleared, coordinates read, rows written
    out = {
        "mode": "cwi",
        "workload": workloads.make_cwi_frame.__doc__.split(":")[0].strip().replace("\n", " "),
        "n": n, "channels": C, "taps": 13, "grid": list(sets[0]["grid"]), "dtype": "f16", "buffer_sets": nsets,
        "build_us": t_build,
        "forward_us": t_fwd,
        "forward_row_order_us": t_fwd_rows,
        "forward_algorithmic_bytes": fwd_bytes,
        "forward_gbs": fwd_bytes / (t_fwd * 1e-6) / 1e9,
        "forward_frac_of_hbm_peak": fwd_bytes / (t_fwd * 1e-6) / 1e9 / HBM_PEAK_GBS,
        "build_algorithmic_bytes": build_bytes,
        "backward_us": t_bwd,
        "backward_algorithmic_bytes": bwd_bytes,
        "backward_gbs": bwd_bytes / (t_bwd * 1e-6) / 1e9,
        "backward_frac_of_hbm_peak": bwd_bytes / (t_bwd * 1e-6) / 1e9 / HBM_PEAK_GBS,
        "graph_replay": not args.no_graph,
    }
    if args.copy_probe:
        copy_probe(torch, dev)
    return out


def bench_xca(torch, sla, workloads, dev, args):
    """The XCA variant, forward and backward, on one frame (Waymo-like by default;
    --config 2, 3 or 4), rows shuffled, plan built outside the timed region,
    beside sla_forward on the same buffers; graph replay over rotated buffer
    sets."""
    cfg = args.config if args.config in (2, 3, 4) else 2
    base = workloads.make_config(cfg, with_grad=False)
    n, H, d, W, dt = base["n"], base["heads"], base["head_dim"], base["num_windows"], base["dtype"]
    tdt = {"f16": torch.float16, "bf16": torch.bfloat16}[dt]
    e = 2
    per_set = 4 * n * H * d * e
    nsets = max(3, int(np.ceil(2 * MALL_BYTES / per_set)) + 1)
    tau = torch.linspace(0.5, 3.0, H, dtype=torch.float32, device=dev)
    sets = []
    for s_ in range(nsets):
        wl = workloads.shuffled(base, [cfg, 2, s_])
        st = {key: torch.from_numpy(np.ascontiguousarray(wl[key])).view(tdt).to(dev) if dt == "bf16"
              else torch.from_numpy(np.ascontiguousarray(wl[key])).to(dev) for key in ("q", "k", "v")}
        st["plan"] = sla.build_segments(torch.from_numpy(wl["ids"]).to(dev), num_windows=W, want_perm=False)
        st["o"] = torch.empty_like(st["q"])
        st["do"] = torch.randn(st["q"].shape, device=dev).to(tdt)
        st["grads"] = [torch.empty_like(st["q"]) for _ in range(3)]
        st["dtau"] = torch.empty(H, dtype=torch.float32, device=dev)
        st["ws"] = torch.empty(sla.lib().sla_xca_backward_workspace_bytes(W, H), dtype=torch.uint8, device=dev)
        sets.append(st)
    torch.cuda.synchronize()

    def timed(fn, reps):
        return time_rotating(torch, dev, fn, sets, reps, args.warmup, eager=args.no_graph)

    reps = max(50, args.steps)
    t_xca = timed(lambda st: sla.forward_xca(st["plan"], st["q"], st["k"], st["v"], tau, out=st["o"]), reps)
    t_sla = timed(lambda st: sla.forward(st["plan"], st["q"], st["k"], st["v"], out=st["o"]), reps)
    t_bwd = timed(lambda st: sla.backward_xca(st["plan"], st["q"], st["k"], st["v"], tau, st["do"], *st["grads"],
                                              dtau=st["dtau"], workspace=st["ws"]), reps)
    nbytes = 4 * n * H * d * e + 4 * n   # q, k, v read and o written once, plus the permutation
    bwd_bytes = 7 * n * H * d * e + 4 * n   # q, k, v, dout read and dq, dk, dv written once, plus the permutation
    return {
        "mode": "xca",
        "workload": base["name"],
        "n": n, "heads": H, "head_dim": d, "num_windows": W, "dtype": dt, "buffer_sets": nsets,
        "xca_us": t_xca,
        "sla_forward_us": t_sla,
        "xca_algorithmic_bytes": nbytes,
        "xca_gbs": nbytes / (t_xca * 1e-6) / 1e9,
        "xca_frac_of_hbm_peak": nbytes / (t_xca * 1e-6) / 1e9 / HBM_PEAK_GBS,
        "xca_backward_us": t_bwd,
        "xca_backward_algorithmic_bytes": bwd_bytes,
        "xca_backward_gbs": bwd_bytes / (t_bwd * 1e-6) / 1e9,
    }


def bench_projected(torch, sla, workloads, dev, args):
    """Projection layer + SLA + output projection on one frame (plan built outside
    the timed region): the fused path against the unfused chain, both timed with
    graph replay over rotated buffer sets."""
    import torch.nn.functional as Fn

    cfg = args.config if args.config in (2, 3, 4) else 2
    base = workloads.make_config(cfg, with_grad=False)
    n, H, d, W, dt = base["n"], base["heads"], base["head_dim"], base["num_windows"], base["dtype"]
    C = H * d
    tdt = {"f16": torch.float16, "bf16": torch.bfloat16}[dt]
    e = 2
    gen = torch.Generator(device="cpu").manual_seed(11)
    w_qkv = (torch.randn(3 * C, C, generator=gen) / C ** 0.5).to(tdt).to(dev)
    b_qkv = (0.1 * torch.randn(3 * C, generator=gen)).to(tdt).to(dev)
    w_o = (torch.randn(C, C, generator=gen) / C ** 0.5).to(tdt).to(dev)
    b_o = (0.1 * torch.randn(C, generator=gen)).to(tdt).to(dev)
    per_set = 6 * n * C * e
    nsets = max(3, int(np.ceil(2 * MALL_BYTES / per_set)) + 1)
    sets = []
    for s_ in range(nsets):
        wl = workloads.shuffled(base, [cfg, 2, s_])
        x = torch.randn(n, C, generator=gen).to(tdt).to(dev)
        plan = sla.build_segments(torch.from_numpy(wl["ids"]).to(dev), num_windows=W, want_perm=False)
        sets.append({"x": x, "plan": plan, "o": torch.empty(n, H, d, dtype=tdt, device=dev),
                     "y": torch.empty(n, C, dtype=tdt, device=dev),
                     "dy": torch.randn(n, C, generator=gen).to(tdt).to(dev),
                     "dx": torch.empty(n, C, dtype=tdt, device=dev),
                     "qkv": torch.empty(3, n, C, dtype=tdt, device=dev)})
    ws = torch.empty(sla.backward_projected_workspace_bytes(n, H, d), dtype=torch.uint8, device=dev)
    torch.cuda.synchronize()

    def fused(st):
        sla.forward_projected(st["plan"], st["x"], w_qkv, w_o, H, b_qkv, b_o, st["o"], st["y"])

    def backward(st):
        sla.backward_projected(st["plan"], st["x"], w_qkv, w_o, st["o"], st["dy"], H, b_qkv, dx=st["dx"],
                               workspace=ws)

    # the forward saving q, k, v, and the backward reading them
    def fused_save(st):
        sla.forward_projected(st["plan"], st["x"], w_qkv, w_o, H, b_qkv, b_o, st["o"], st["y"],
                              qkv_out=st["qkv"])

    def backward_saved(st):
        sla.backward_projected(st["plan"], st["x"], w_qkv, w_o, st["o"], st["dy"], H, b_qkv, dx=st["dx"],
                               workspace=ws, qkv=st["qkv"])

    def unfused(st):
        qkv = Fn.linear(st["x"], w_qkv, b_qkv)
        q, k, v = (qkv[:, i * C:(i + 1) * C].contiguous().view(n, H, d) for i in range(3))
        o = sla.forward(st["plan"], q, k, v, out=st["o"])
        st["y"].copy_(Fn.linear(o.view(n, C), w_o, b_o))

    def timed(fn, reps):
        return time_rotating(torch, dev, fn, sets, reps, args.warmup, eager=args.no_graph)

    reps = max(50, args.steps)
    t_fused = timed(fused, reps)
    t_unfused = timed(unfused, reps)
    for st in sets:     # the forward's o of every set, for the backward
        fused(st)
    t_backward = timed(backward, reps)
    t_fused_save = timed(fused_save, reps)
    for st in sets:     # the saved q, k, v of every set
        fused_save(st)
    t_backward_saved = timed(backward_saved, reps)
    fused_bytes = 4 * n * C * e     # x read, o written; o read, y written
    unfused_bytes = 10 * n * C * e  # + q, k, v written and read, and their copies' extra pass
    # backward, least traffic: x, o, dy read and dx written (q, k, v, do, dq, dk, dv
    # are intermediates), plus the SLA backward's own 7 n C e
    backward_bytes = (4 + 7) * n * C * e
    return {
        "mode": "projected",
        "workload": base["name"],
        "n": n, "heads": H, "head_dim": d, "dtype": dt, "buffer_sets": nsets,
        "fused_us": t_fused,
        "unfused_us": t_unfused,
        "speedup": t_unfused / t_fused,
        "fused_algorithmic_bytes": fused_bytes,
        "fused_gbs": fused_bytes / (t_fused * 1e-6) / 1e9,
        "fused_frac_of_hbm_peak": fused_bytes / (t_fused * 1e-6) / 1e9 / HBM_PEAK_GBS,
        "unfused_chain": "torch linear (x W_qkv^T + b), three contiguous q/k/v copies, sla_forward, "
                         "torch linear (o W_o^T + b)",
        "backward_us": t_backward,
        "backward_algorithmic_bytes": backward_bytes,
        "backward_gbs": backward_bytes / (t_backward * 1e-6) / 1e9,
        "backward_frac_of_hbm_peak": backward_bytes / (t_backward * 1e-6) / 1e9 / HBM_PEAK_GBS,
        "backward_path": "sla_backward_projected: q, k, v recomputed, do, SLA backward, dx, "
                         "weight and bias gradients (fp32, fixed-order sums)",
        "fused_save_us": t_fused_save,
        "backward_saved_us": t_backward_saved,
        "saved_qkv_path": "the forward also stores q, k, v (3 n C e bytes more), the backward reads them "
                          "instead of recomputing them",
        "train_pair_us": t_fused + t_backward,
        "train_pair_saved_us": t_fused_save + t_backward_saved,
    }


def compare_scatter(torch, sla, workloads, dev):
    """Forward of the chunk-wise path (sla_forward) against the naive scatter-based
    one (sla_forward_scatter: a cached kv matrix per voxel, summed per window), the
    comparison of the paper's Fig. 4, on fp16 inputs with H = 4, d = 32:
      * sequence length: 1, 2, 4 and 8 Waymo-like frames concatenated;
      * window length: about 131k voxels in equal windows of 16 .. 1024 rows.
    Each case: median of 20 timed calls (HIP events, inputs resident) after 3
    warm-up calls; memory = the plan (chunk-wise) or the kv cache (scatter)."""
    H, d = 4, 32

    def time_call(fn, reps=20):
        for _ in range(3):
            fn()
        torch.cuda.synchronize()
        ts = []
        for _ in range(reps):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            fn()
            b.record()
            torch.cuda.synchronize()
            ts.append(a.elapsed_time(b) * 1e3)
        return float(np.median(ts))

    def case(ids, W, label):
        rng = np.random.default_rng([99, ids.size])
        n = ids.size
        q, k, v = (torch.from_numpy(workloads.normal_values(rng, n, H, d, "f16")).to(dev)
                   for _ in range(3))
        plan = sla.build_segments(torch.from_numpy(ids).to(dev), num_windows=W)
        o1, o2 = torch.empty_like(q), torch.empty_like(q)
        ws = torch.empty(sla.scatter_workspace_bytes(n, H, d), dtype=torch.uint8, device=dev)
        t_chunk = time_call(lambda: sla.forward(plan, q, k, v, out=o1))
        t_scat = time_call(lambda: sla.forward_scatter(plan, q, k, v, out=o2, workspace=ws))
        diff = float((o1.float() - o2.float()).abs().max() / o2.float().abs().max())
        out = {"case": label, "n": n, "windows": W, "chunkwise_us": t_chunk, "scatter_us": t_scat,
               "speedup": t_scat / t_chunk, "chunkwise_extra_bytes": sla.plan_bytes(n, W),
               "scatter_extra_bytes": int(ws.numel()), "max_rel_diff": diff}
        del ws, q, k, v, o1, o2
        torch.cuda.synchronize()
        return out

    rows = []
    for frames in (1, 2, 4, 8):
        ids = np.concatenate([workloads.waymo_like_ids(np.random.default_rng([6, 0, f])) +
                              f * workloads.FRAME_WINDOWS for f in range(frames)]).astype(np.int32)
        rows.append(case(ids, frames * workloads.FRAME_WINDOWS, f"{frames} frame(s)"))
    for wlen in (16, 64, 144, 512, 1024):
        nw = 131072 // wlen
        ids = workloads.ids_from_lengths(np.full(nw, wlen), np.random.default_rng([7, wlen]))
        rows.append(case(ids, nw, f"windows of {wlen} rows"))
    return {"metric": "SLA forward: chunk-wise vs naive scatter-based (time and extra memory)",
            "dtype": "f16", "heads": H, "head_dim": d, "data": "synthetic", "comparison": rows}


def copy_probe(torch, dev):
    """Three plain device-to-device copies of COPY_PROBE_BYTES from distinct
    buffers: the reference dispatches that scale the HBM byte counters."""
    for _ in range(3):
        a = torch.empty(COPY_PROBE_BYTES, dtype=torch.uint8, device=dev).fill_(1)
        b = torch.empty_like(a)
        torch.cuda.synchronize()
        b.copy_(a)
        torch.cuda.synchronize()
        del a, b


def measure_copy(torch, dev, nbytes=COPY_PROBE_BYTES, reps=5):
    """GB/s (read + write bytes) of a plain device-to-device copy of `nbytes`,
    buffers rotated so that the Infinity Cache cannot serve repeats."""
    bufs = [torch.empty(nbytes, dtype=torch.uint8, device=dev).fill_(1) for _ in range(3)]
    dst = torch.empty_like(bufs[0])
    dst.copy_(bufs[0])
    torch.cuda.synchronize()
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0.record()
    for i in range(reps):
        dst.copy_(bufs[i % 3])
    t1.record()
    torch.cuda.synchronize()
    ms = t0.elapsed_time(t1) / reps
    del bufs, dst
    return 2 * nbytes / (ms * 1e-3) / 1e9


def measure_gather(torch, dev, sets, perms, names, reps=20):
    """GB/s (read + write bytes) of torch's row gather (index_select through each
    set's plan permutation into contiguous rows) over the matrices `names` of the
    rotating buffer sets, in one graph: what a library gather reaches on the
    same rows in the same order, for scale.  None without permutations."""
    if perms is None:
        return None
    idx = [p.long() for p in perms]
    outs = [[torch.empty_like(st[m]) for m in names] for st in sets]
    def run():
        for st, ix, o in zip(sets, idx, outs):
            for m, dst in zip(names, o):
                torch.index_select(st[m], 0, ix, out=dst)
    run()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    cap = torch.cuda.Stream(dev)
    cap.wait_stream(torch.cuda.current_stream(dev))
    with torch.cuda.stream(cap):
        with torch.cuda.graph(g, stream=cap):
            run()
    torch.cuda.current_stream(dev).wait_stream(cap)
    g.replay()
    torch.cuda.synchronize()
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0.record()
    for _ in range(reps):
        g.replay()
    t1.record()
    torch.cuda.synchronize()
    ms = t0.elapsed_time(t1) / reps
    nbytes = sum(2 * st[m].numel() * st[m].element_size() for st in sets for m in names)
    del g, outs
    return nbytes / (ms * 1e-3) / 1e9


def cpu_model():
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


# ---- the oracle on every host core: a process pool over contiguous window ranges
_POOL_WL = {}


def _pool_init(cfg, training):
    import workloads
    import oracle

    wl = workloads.make_config(cfg, with_grad=training)
    dt = wl["dtype"]
    _POOL_WL["q"], _POOL_WL["k"], _POOL_WL["v"] = (oracle.widen(wl[x], dt) for x in ("q", "k", "v"))
    _POOL_WL["do"] = oracle.widen(wl["dout"], dt) if training else None


def _pool_work(job):
    """The oracle on one contiguous range of windows: the range's rows (in window
    order) with offsets local to them, a scene of its own."""
    import oracle

    rows, off, training, variant = job
    extra = () if variant is None else variant
    w = _POOL_WL
    q, k, v = w["q"][rows], w["k"][rows], w["v"][rows]
    oracle.sla_forward_ref(q, k, v, off, None, *extra)
    if training:
        oracle.sla_backward_ref(q, k, v, w["do"][rows], off, None, *extra)
    return int(rows.size)


def cpu_baseline_pool(cfg, training, budget_s, variant=None, max_procs=16):
    """The same oracle calls split over contiguous window ranges of balanced row
    counts, one range per process (at most 16: one GPU's share of the host); the
    segment build runs in the parent.  Workers start (and build their inputs)
    before the clock starts."""
    import multiprocessing as mp

    import oracle
    import workloads

    procs = max(1, min(max_procs, len(os.sched_getaffinity(0))))
    base = workloads.make_config(cfg, with_grad=False)
    old = {k: os.environ.get(k) for k in ("OMP_NUM_THREADS", "OPENBLAS_NUM_THREADS", "MKL_NUM_THREADS")}
    for k in old:
        os.environ[k] = "1"
    try:
        ctx = mp.get_context("spawn")
        with ctx.Pool(procs, initializer=_pool_init, initargs=(cfg, training)) as pool:
            def one():
                if base["ids"] is not None:
                    perm, off, _ = oracle.segments_ref(base["ids"], base["num_windows"])
                else:
                    perm, off = None, base["offsets"].astype(np.int64)
                W = len(off) - 1
                cuts = np.searchsorted(off, np.linspace(0, off[-1], procs + 1)).clip(0, W)
                cuts[0], cuts[-1] = 0, W
                order = perm if perm is not None else np.arange(off[-1])
                jobs = [(order[off[a]:off[b]], off[a:b + 1] - off[a], training, variant)
                        for a, b in zip(cuts[:-1], cuts[1:]) if b > a]
                assert sum(pool.map(_pool_work, jobs)) == off[-1]
            one()                                   # untimed: workers warm
            reps, t_start = 0, time.perf_counter()
            while True:
                one()
                reps += 1
                if time.perf_counter() - t_start >= budget_s:
                    break
            el = time.perf_counter() - t_start
    finally:
        for k, v in old.items():
            if v is None:
                os.environ.pop(k, None)
            else:
                os.environ[k] = v
    per = el / reps
    return {
        "value": base["n"] / per,
        "unit": "voxels/s",
        "cores": procs,
        "kind": "oracle",
        "sample": f"{reps} whole frame(s), windows split over {procs} processes, {el:.1f} s wall",
        "ms_per_frame": per * 1e3,
    }


def cpu_baseline(base, training, budget_s, variant=None):
    """The CPU oracle as it stands, on whole frames of the same workload."""
    import oracle

    try:
        from threadpoolctl import threadpool_limits
    except ImportError:  # pragma: no cover
        threadpool_limits = None
    dt = base["dtype"]
    q, k, v = (oracle.widen(base[x], dt) for x in ("q", "k", "v"))
    do = oracle.widen(base["dout"], dt) if training else None

    def one():
        if base["ids"] is not None:
            perm, off, _ = oracle.segments_ref(base["ids"], base["num_windows"])
        else:
            perm, off = None, base["offsets"].astype(np.int64)
        extra = () if variant is None else variant
        oracle.sla_forward_ref(q, k, v, off, perm, *extra)
        if training:
            oracle.sla_backward_ref(q, k, v, do, off, perm, *extra)

    ctx = threadpool_limits(limits=1) if threadpool_limits else None
    if ctx:
        ctx.__enter__()
    try:
        reps, t_start = 0, time.perf_counter()
        while True:
            one()
            reps += 1
            if time.perf_counter() - t_start >= budget_s:
                break
        el = time.perf_counter() - t_start
    finally:
        if ctx:
            ctx.__exit__(None, None, None)
    per = el / reps
    return {
        "value": base["n"] / per,
        "unit": "voxels/s",
        "cores": 1,
        "kind": "oracle",
        "cpu_model": cpu_model(),
        "sample": f"{reps} whole frame(s) of N={base['n']} voxels, "
                  f"{'segments+forward+backward' if training else 'segments+forward'} in numpy float64, "
                  f"{el:.1f} s wall, 1 thread",
        "ms_per_frame": per * 1e3,
    }


if __name__ == "__main__":
    main()
