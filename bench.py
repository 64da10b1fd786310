#!/usr/bin/env python3
"""Benchmark of the sparse contact-layer path on one MI355X.

One step = one pass of the whole path over one batch of synthetic input:

    mask compaction (+ neighbour-row table of the active set) -> gather of the
    active rows -> sparse linear + ReLU -> sparse 9-slot neighbourhood conv +
    ReLU -> zero-fill scatter + per-body max-pool

on the density-sweep workload at 5% density: B = 128 bodies, V = 10475 mesh
vertices (ellipsoid, exact 9-NN), C = 128 bf16 channels, i.i.d. Bernoulli(0.05)
mask.  `value` is active-vertex rows per second per sparse layer over the whole
step: N' * (number of sparse layers) / step time, with every input resident in
HBM when the timed region starts.  The line also carries the roofline of the
dominant kernel (HIP events on the stream it runs on), the speed-up of each
sparse layer over the same layer run densely on all B*V rows, and the CPU
oracle timed on a bounded sample of the same workload.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-cpu-baseline]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
BF16_MFMA_PEAK_TFLOPS = 2500.0
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_sparse_conv_c4_5pct.txt")
# sources of the conv launch (dispatch and kernel): the counter summary is
# only used while they are unchanged
EVENT_EVERY = 50  # steps between two sampled conv launches in the timed region
KERNEL_SOURCES = [os.path.join(ROOT, "paper_2608_09388_amd", "csrc", f)
                  for f in ("conv_packed.hip", "gemm.hip", "conv_ws.hip", "conv_sm.hip",
                            "shc_internal.h")]


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=1000)
    p.add_argument("--warmup", type=int, default=50)
    p.add_argument("--density", type=float, default=0.05)
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-dense", action="store_true", help="skip the dense-layer comparison")
    p.add_argument("--no-sweep", action="store_true",
                   help="skip the density sweep and the full-mesh layers")
    p.add_argument("--step-only", action="store_true",
                   help="the step, its per-kernel times and roofline only (one workload, "
                        "for kernel traces of the density-sweep batch alone)")
    p.add_argument("--stacks-only", action="store_true",
                   help="only the other configurations' stacks (config_stacks), with --steps, "
                        "--warmup and --reps (for kernel traces of the split conv)")
    p.add_argument("--cpu-seconds", type=float, default=15.0)
    p.add_argument("--reps", type=int, default=50,
                   help="back-to-back launches per kernel for the per-kernel times")
    p.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                   help="only run a plain device copy of MIB MiB (counter calibration) and exit")
    return p.parse_args()


def algorithmic_conv(w, coords, inv, n, e, layer=1):
    """Bytes and useful flops the conv (layer `layer`) must move/do for N'
    rows (per launch)."""
    K, Cin, Cout = w.layers[layer].W.shape
    b = coords[:, 0].astype(np.int64)
    v = coords[:, 1].astype(np.int64)
    present = 0
    for j in range(K):
        u = w.nbr[v, j].astype(np.int64)
        present += int(np.count_nonzero((u >= 0) & (inv[b * w.V + np.maximum(u, 0)] >= 0)))
    bytes_ = (present * Cin * e        # present neighbour rows read
              + n * 4 * K              # neighbour-row table entries
              + n * Cout * e           # output rows
              + K * Cin * Cout * e)    # weights once
    flops = 2.0 * present * Cin * Cout
    return bytes_, flops, present / (n * K)


def algorithmic_step_bytes(w, n, e, conv_bytes):
    """Bytes each kernel of the step must move for N' = n active rows, from
    the per-unit figures of the path (Sec. 3 operators): compaction reads the
    mask byte and writes the inverse-map entry of every dense vertex, plus a
    coordinate pair per active row and an offset per body; the neighbour-row
    table reads a coordinate pair and K neighbour and inverse-map entries and
    writes K table entries per row (K neighbour entries and K table entries
    when the compaction writes it, the row numbering staying on chip); the
    fused gather + linear reads a
    coordinate pair and C_in features and writes C_out per row, plus the
    weights once; the zero-fill scatter reads each active row and writes
    every dense row (reading its inverse-map entry); the pool reads each
    active row and writes a row per body (reading its offset)."""
    B, V, K = w.B, w.V, w.K
    Cin, Cout = w.layers[0].W.shape[-2:]
    C = w.layers[-1].W.shape[-1]
    BV = B * V
    return {
        "compact": BV * (1 + 4) + n * 8 + (B + 1) * 4,
        "table": n * (8 + 3 * 4 * K),
        # in one pass: the table reads only the neighbour lists
        "compact+table": BV * (1 + 4) + n * 8 + (B + 1) * 4 + n * 2 * 4 * K,
        "gather+linear": n * (8 + Cin * e + Cout * e) + Cin * Cout * e,
        "conv": conv_bytes,
        "scatter": n * C * e + BV * (4 + C * e),
        "pool": n * C * e + B * (4 + C * e),
    }


def kernel_source_digest():
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        h.update(open(f, "rb").read())
    return h.hexdigest()


def traffic_from_profile():
    """HBM bytes per conv launch from the committed rocprofv3 counter summary,
    or None if absent or taken on a different version of the kernel source."""
    if not os.path.exists(TRAFFIC_FILE):
        return None
    kv = {}
    for line in open(TRAFFIC_FILE):
        if ":" in line and not line.lstrip().startswith("#"):
            k, v = line.split(":", 1)
            kv[k.strip()] = v.strip()
    src = kernel_source_digest()
    if kv.get("kernel_source_sha256") != src or "hbm_bytes_per_launch" not in kv:
        return None
    return float(kv["hbm_bytes_per_launch"])


def cpu_model():
    """The host CPU's model name (first 'model name' line of /proc/cpuinfo)."""
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(w, layers_spec, budget_s):
    """The oracle as it stands on a bounded sample of bodies of the same
    workload: one warm-up run, then the median of three timed runs, once with
    the BLAS pool on every core this process may use and once limited to one
    thread (threadpoolctl), each on its own body sample sized for about
    budget_s / 8 seconds per run."""
    import threadpoolctl
    from oracle import shc_oracle as O

    def run(nb):
        t = time.perf_counter()
        r = O.run_stack(w.x[: nb * w.V], w.mask[:nb], w.nbr, layers_spec, w.dtype, pool=True)
        O.scatter(r["outs"][-1], r["inv"], zero_fill=True)
        return time.perf_counter() - t, r["n"]

    def leg(threads):
        with threadpoolctl.threadpool_limits(limits=threads):
            t1, _ = run(1)                                  # sizing run
            nb = int(max(1, min(w.B, budget_s / 8 / max(t1, 1e-3))))
            run(nb)                                         # warm-up
            times = []
            for _ in range(3):
                t, n = run(nb)
                times.append(t)
        t = float(np.median(times))
        return nb, n, t, n * len(layers_spec) / t

    affinity = len(os.sched_getaffinity(0))
    nb, n, t, rate = leg(affinity)
    nb1, n1, t1, rate1 = leg(1)
    return {"value": rate, "unit": "active-vertex rows/s per sparse layer",
            "cores": affinity, "kind": "oracle",
            "sample": (f"{nb} of {w.B} bodies ({n} active rows), full step; median of 3 runs "
                       f"after a warm-up, {t:.2f} s each; fp64 numpy"),
            "value_1thread": rate1,
            "sample_1thread": (f"{nb1} of {w.B} bodies ({n1} active rows), median of 3 after "
                               f"a warm-up, {t1:.2f} s each"),
            "nproc": os.cpu_count(), "cpu_model": cpu_model(),
            "paper_context": ("the paper reports 0.009 s per sample for its whole network on one "
                              "NVIDIA Tesla V100, 12 times faster than the next-best method, and "
                              "0.28 s -> 0.009 s when one mask cuts the processed vertices from "
                              "655 to 66 (Table 4); a whole-model latency on other hardware, not "
                              "comparable with this per-layer throughput")}


def kernel_times(st, shc, torch, reps):
    """Average duration of each kernel of the path: `reps` launches back to
    back on the stream each call uses, bracketed by two HIP events there."""
    main = torch.cuda.current_stream()
    n = st.n

    def compact_async():  # compaction without the host count (no sync per call)
        shc.compact_mask(st.mask, st.B, st.V, st.coords, st.inv, st.row_ptr, st.n_active, st.ws,
                         want_host_count=False)

    calls = {"compact": (compact_async, main), "table": (st.build_table, main),
             # the step's compaction: with the table written in the same pass
             # when the set is built that way (no host wait: start only)
             "compact+table": (st._set.compact.start, main),
             "gather": (st.gather, main),
             ("gather+linear" if st.fused_gather else "linear"): (lambda: st.layer(0), main),
             "conv": (lambda: st.layer(1), main), "scatter": (st.scatter, main),
             "pool": (st.pool, main)}
    if st.fused_gather:  # the step has no separate gather kernel
        del calls["gather"]
    if not st._set.fused:
        del calls["compact+table"]
    out = {}
    for name, (fn, stream) in calls.items():
        for _ in range(3):
            fn()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        a.record(stream)
        for _ in range(reps):
            fn()
        b.record(stream)
        torch.cuda.synchronize()
        out[name] = a.elapsed_time(b) / reps
    st.n = n
    return out


def copy_calibration(torch, mib):
    """A plain device-to-device copy of `mib` MiB, five times: the reference
    for scaling the FETCH_SIZE / WRITE_SIZE counters to bytes."""
    n = mib * 1024 * 1024 // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda:0")
    dst = torch.empty_like(src)
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_mib": mib, "copies": 5}))


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only; --gpus {args.gpus} is not supported "
              "(the path is single-GPU; sharding across GPUs is described, not built)",
              file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2608_09388_amd import binding as shc
    from paper_2608_09388_amd import synth
    from paper_2608_09388_amd.pipeline import SparseStack

    shc.load()
    if args.copy_calibration:
        copy_calibration(torch, args.copy_calibration)
        return
    if args.stacks_only:
        print(json.dumps({"config_stacks": config_stacks_measure(
            torch, steps=args.steps, warmup=args.warmup, reps=args.reps)}))
        return
    w = synth.workload_c4(args.density)
    # the next batch's compaction and neighbour table run on a second stream
    # beside the current batch's scatter and pool
    st = SparseStack(w, device="cuda:0", side_stream=True)
    n = st.compact()
    log(f"workload ready: N'={n} active rows of {w.B * w.V}")
    L = len(w.layers)
    stream = torch.cuda.current_stream()

    st.run(args.warmup)
    torch.cuda.synchronize()

    # timed region: K whole steps over consecutive batches (each step's
    # compaction and table on the side stream, overlapped with the previous
    # step's scatter and pool); HIP
    # events around the conv launch of every EVENT_EVERY-th step, on the
    # stream it runs on (a pair of timing events costs the step a few us)
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          if k % EVENT_EVERY == 0 else (None, None) for k in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    st.run(args.steps, around_layer=(1, ev))
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_per_step = wall * 1e3 / args.steps
    conv_in_step_ms = float(np.mean([a.elapsed_time(b) for a, b in ev if a is not None]))
    log(f"timed {args.steps} steps: {ms_per_step:.4f} ms/step")
    value = n * L / (ms_per_step / 1e3)

    per_kernel_ms = kernel_times(st, shc, torch, args.reps)
    log("per-kernel times done")

    # roofline of the dominant kernel (the conv layer)
    coords = st.coords[:n].cpu().numpy()
    inv = st.inv.cpu().numpy()
    e = 2
    cbytes, cflops, a_present = algorithmic_conv(w, coords, inv, n, e)
    # kernel duration: back-to-back launches on the conv's stream (the in-step
    # events also hold the dispatch gap before the launch); rocprofv3's average
    # kernel duration agrees with this figure
    conv_s = per_kernel_ms["conv"] / 1e3
    ridge = BF16_MFMA_PEAK_TFLOPS * 1e12 / (HBM_PEAK_GBS * 1e9)
    traffic = traffic_from_profile()
    if cflops / cbytes < ridge:
        ach = cbytes / conv_s / 1e9
        roof = {"bound": "hbm", "achieved": round(ach, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(ach / HBM_PEAK_GBS, 4), "traffic": traffic}
    else:
        ach = cflops / conv_s / 1e12
        roof = {"bound": "mfma", "achieved": round(ach, 2), "peak": BF16_MFMA_PEAK_TFLOPS,
                "unit": "TFLOP/s", "frac": round(ach / BF16_MFMA_PEAK_TFLOPS, 4),
                "traffic": traffic}
    roof["kernel"] = ("shc_sparse_neighbor_conv_packed (conv_packed_kernel: every slot's "
                      "weights in registers, one chunk of active rows per CU, rows grouped by "
                      "their slots in LDS)"
                      if max(1, st.packed_min_rows) <= n <= st.packed_rows.get(1, 0) else
                      "shc_sparse_neighbor_conv_table (ws_kernel: weight slice resident in "
                      "LDS, index sets from the neighbour-row table)")
    roof["algorithmic_bytes"] = int(cbytes)
    roof["useful_flops"] = cflops
    roof["executed_slot_gemm_flops"] = 2.0 * n * 9 * 128 * 128
    roof["present_slot_fraction"] = round(a_present, 4)
    roof["launch_us"] = round(per_kernel_ms["conv"] * 1e3, 2)
    roof["launch_us_in_step_events"] = round(conv_in_step_ms * 1e3, 2)

    # every kernel of the step against HBM: algorithmic bytes / back-to-back
    # duration (compaction and table are latency-bound at this size)
    step_bytes = algorithmic_step_bytes(w, n, e, cbytes)
    kernel_rooflines = {}
    for name, b in step_bytes.items():
        if name in per_kernel_ms:
            t = per_kernel_ms[name] / 1e3
            kernel_rooflines[name] = {"algorithmic_bytes": int(b), "us": round(t * 1e6, 2),
                                      "GB/s": round(b / t / 1e9, 1),
                                      "frac_hbm": round(b / t / 1e9 / HBM_PEAK_GBS, 4)}

    out = {
        "metric": "active-vertex rows/sec per sparse contact layer; speed-up vs dense layer",
        "value": round(value, 1),
        "unit": "active-vertex rows/s per sparse layer",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic",
        "config": {"workload": f"density sweep point p={args.density:g}: B=128 bodies, "
                               f"V=10475 ellipsoid mesh, K=9 exact kNN, C=128->128 bf16, "
                               f"sparse linear + sparse conv (+ReLU), scatter + max-pool",
                   "B": w.B, "V": w.V, "K": w.K, "C": 128, "density": args.density,
                   "n_active": n, "sparse_layers": L, "parallelism": "single GPU"},
        "per_kernel_us": {k: round(v * 1e3, 2) for k, v in per_kernel_ms.items()},
        "roofline": roof,
        "kernel_rooflines": kernel_rooflines,
    }

    # the step's kernels back to back, against the pipelined step; and the
    # per-layer rate (N' / one layer's launch)
    sum_keys = ["compact+table" if "compact+table" in per_kernel_ms else "compact",
                "gather+linear", "conv", "scatter", "pool"]
    ksum = sum(per_kernel_ms[k] for k in sum_keys if k in per_kernel_ms)
    out["step_breakdown"] = {
        "kernels": sum_keys, "kernel_sum_us": round(ksum * 1e3, 2),
        "step_over_kernel_sum": round(ms_per_step / ksum, 4),
        "per_layer_rows_per_s": {
            "gather+linear": round(n / (per_kernel_ms["gather+linear"] / 1e3), 1),
            "conv": round(n / (per_kernel_ms["conv"] / 1e3), 1)}}
    if args.step_only:
        print(json.dumps(out))
        return
    out["chains"] = chain_measure(w, torch, args.steps, args.warmup)
    log("scatter-only and pool-only chains measured")
    out["config_stacks"] = config_stacks_measure(torch)
    log("the other configurations' stacks measured")
    out["gather_scatter"] = gather_scatter_measure(shc, synth, torch, args.reps)
    log("gather and scatter measured")
    out["cold_warm"] = cold_warm_measure(st, torch)
    log("cold and warm launches measured")
    out["conv_plan"] = conv_plan_measure(st, shc, torch, args.reps)
    log("conv plan measured")
    out["incremental_scatter"] = incremental_scatter_measure(w, shc, synth, torch, args.reps)
    log("incremental scatter measured")
    out["measured_peaks"] = measured_peaks(torch)
    log("measured peaks done")
    if not args.no_sweep:
        out["density_sweep"] = density_sweep(w, shc, synth, torch, args.reps)
        log("density sweep measured")
        out["c3_layers"] = c3_layers(shc, synth, torch, args.reps)
        log("full-mesh layers measured")
    out["next_rows"] = {"group_norm": group_norm_measure(st, shc, torch, args.reps),
                        "multi_mask": multi_mask_measure(st, w, shc, synth, torch, args.reps),
                        "mask_scores": mask_scores_measure(w, shc, torch, args.reps),
                        "backward": backward_measure(st, w, shc, torch, args.reps)}
    log("group norm measured")

    if not args.no_dense:
        out["speedup_vs_dense"] = dense_comparison(st, w, per_kernel_ms, torch, shc, synth)
        log("dense comparison done")
    if not args.no_cpu_baseline:
        spec = [(l.kind, l.W, l.bias, l.relu) for l in w.layers]
        out["cpu_baseline"] = cpu_baseline(w, spec, args.cpu_seconds)
        log("cpu baseline done")
    print(json.dumps(out))


def measured_peaks(torch, reps=20):
    """What this GPU reaches on plain work, beside the published peaks: a
    device-to-device copy of 1 GiB (PyTorch's copy kernel; read + write bytes
    over its time) and an 8192^3 bf16 GEMM (PyTorch's matmul, hipBLASLt)."""
    n = 1 << 29                                   # 1 GiB of bf16
    x = torch.empty(n, dtype=torch.bfloat16, device="cuda:0").normal_()
    y = torch.empty_like(x)
    t_copy = _time_us(lambda: y.copy_(x), torch, reps)
    copy_gbs = 2 * n * 2 / (t_copy * 1e-6) / 1e9
    del x, y
    m = 8192
    a = torch.randn((m, m), device="cuda:0").to(torch.bfloat16)
    b = torch.randn((m, m), device="cuda:0").to(torch.bfloat16)
    t_mm = _time_us(lambda: torch.mm(a, b), torch, reps)
    tflops = 2.0 * m ** 3 / (t_mm * 1e-6) / 1e12
    del a, b
    torch.cuda.empty_cache()
    return {"copy_1GiB_GBs": round(copy_gbs, 1), "copy_frac_of_peak": round(copy_gbs / HBM_PEAK_GBS, 4),
            "gemm_bf16_8192_TFLOPs": round(tflops, 1),
            "gemm_frac_of_peak": round(tflops / BF16_MFMA_PEAK_TFLOPS, 4)}


def conv_plan_measure(st, shc, torch, reps):
    """The conv layer of the step from its table against the same layer from
    a plan of the active set (index lists, sort and job lists built once by
    shc_build_conv_plan): the plan build, a planned layer, and three layers
    of that shape chained on the set -- from the table each, or one build
    and three planned layers.  Back-to-back prepared calls between HIP
    events; outputs checked equal."""
    n = st.n
    W, bias = st.weights[1], st.biases[1]
    K, Cin, Cout = W.shape
    nb = shc.conv_plan_bytes(n, K, Cin, Cout)
    if nb == 0:
        return {"config": f"N'={n}: no plan for this row count"}
    plan = torch.empty(nb, dtype=torch.uint8, device=st.device)
    src = st.acts[1]
    y = [torch.empty((n, Cout), dtype=src.dtype, device=st.device) for _ in range(4)]
    build = shc.prepare_build_conv_plan(st.table, K, Cin, Cout, plan)
    tab = [shc.prepare_sparse_neighbor_conv_table(a, st.table, W, bias, b)
           for a, b in ((src, y[0]), (y[0], y[1]), (y[1], y[2]))]
    pl = [shc.prepare_sparse_neighbor_conv_planned(a, plan, W, bias, b)
          for a, b in ((src, y[3]), (y[3], y[1]), (y[1], y[2]))]
    build(n)
    tab[0](n)
    pl[0](n)
    torch.cuda.synchronize()
    same = bool(torch.equal(y[0], y[3]))
    t_tab = _time_us(lambda: tab[0](n), torch, reps)
    t_build = _time_us(lambda: build(n), torch, reps)
    t_pl = _time_us(lambda: pl[0](n), torch, reps)
    t_tab3 = _time_us(lambda: [c(n) for c in tab], torch, reps)
    t_pl3 = _time_us(lambda: (build(n), [c(n) for c in pl]), torch, reps)
    return {"config": f"N'={n} rows of the density-sweep set, K={K}, C={Cin}->{Cout} bf16, "
                      f"plan {nb} bytes",
            "planned_equals_table": same, "table_conv_us": round(t_tab, 2),
            "plan_build_us": round(t_build, 2), "planned_conv_us": round(t_pl, 2),
            "three_layers_table_us": round(t_tab3, 2),
            "three_layers_build_and_planned_us": round(t_pl3, 2)}


def config_stacks_measure(torch, steps=500, warmup=30, reps=50):
    """The other configurations' whole stacks (the tiny fp32 layer, the
    4-layer encoder, the sequence workload), pipelined as the headline step:
    ms per step, rows/s per sparse layer, each layer's launch on its own
    (back to back between HIP events) and which conv kernel it ran; a layer
    that runs as the split conv is also timed as the table conv."""
    from paper_2608_09388_amd import binding as shc
    from paper_2608_09388_amd import synth
    from paper_2608_09388_amd.pipeline import SparseStack
    out = []
    for name, mk in (("tiny spiral-conv layer", synth.workload_c1),
                     ("4-layer encoder", synth.workload_c2),
                     ("sequences", synth.workload_c5)):
        w = mk()
        st = SparseStack(w, device="cuda:0", side_stream=True)
        n = st.compact()
        st.run(warmup)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        st.run(steps)
        torch.cuda.synchronize()
        ms = (time.perf_counter() - t0) * 1e3 / steps
        n = st.n
        if st.table is not None:
            st.build_table()
        layer_us = [round(_time_us(lambda l=l: st.layer(l), torch, reps), 2)
                    for l in range(len(w.layers))]
        kinds = []
        for l, spec in enumerate(w.layers):
            if spec.kind != "conv":
                kinds.append("linear")
            elif max(1, st.packed_min_rows) <= n <= st.packed_rows.get(l, 0):
                kinds.append("packed conv")
            elif 0 < n <= st.split_rows.get(l, 0):
                kinds.append("split conv")
            elif 0 < n <= st.plan_shapes.get(tuple(st.weights[l].shape), 0):
                kinds.append("planned conv")
            else:
                kinds.append("table conv")
        # the split layers' table conv on the same rows, for comparison
        table_us = {}
        for l, kind in enumerate(kinds):
            if kind == "split conv":
                tmp = torch.empty_like(st.acts[l + 1][:max(n, 1)])
                call = shc.prepare_sparse_neighbor_conv_table(st.acts[l], st.table, st.weights[l],
                                                              st.biases[l], tmp)
                table_us[l] = round(_time_us(lambda c=call: c(n), torch, reps), 2)
                del tmp
        out.append({"workload": w.name, "dtype": w.dtype, "B": w.B, "V": w.V, "n_active": n,
                    "layers": [f"{l.kind} {l.Cin}->{l.Cout}" for l in w.layers],
                    "layer_kernels": kinds,
                    "split_layers_table_conv_us": table_us,
                    "ends_in": ("scatter" if w.scatter else "") + (" pool" if w.pool else ""),
                    "ms_per_step": round(ms, 4),
                    "rows_per_s_per_layer": round(n * len(w.layers) / (ms / 1e3), 1),
                    "layer_us": layer_us,
                    "layer_rows_per_s": [round(n / (u * 1e-6), 1) for u in layer_us]})
        del st
    return out


def chain_measure(w, torch, steps, warmup):
    """The same pipelined step ending in the scatter alone or the pool alone
    (the path ends in "a scatter or a segmented pool"; the headline step does
    both): ms per step and rows/s per sparse layer for each ending."""
    import dataclasses
    from paper_2608_09388_amd.pipeline import SparseStack
    res = {}
    for name, scatter, pool in (("scatter_only", True, False), ("pool_only", False, True)):
        wv = dataclasses.replace(w, scatter=scatter, pool=pool)
        st = SparseStack(wv, device="cuda:0", side_stream=True)
        n = st.compact()
        st.run(warmup)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        st.run(steps)
        torch.cuda.synchronize()
        ms = (time.perf_counter() - t0) * 1e3 / steps
        res[name] = {"ms_per_step": round(ms, 4),
                     "rows_per_s_per_layer": round(n * len(w.layers) / (ms / 1e3), 1)}
        del st
    return res


def incremental_scatter_measure(w, shc, synth, torch, reps, steps=300, warmup=30):
    """The zero-fill scatter against shc_scatter_update on consecutive batches
    whose masks differ: two independent Bernoulli(p) masks of the density-
    sweep workload, alternated.  The update kernel alone (back to back,
    A -> B then B -> A, each checked equal to the zero-fill scatter of its
    set), and the whole step with either scatter when the masks alternate
    (the mask of each batch copied into place on the device first, in both
    runs).  Algorithmic bytes of an update: the current rows read and written
    (2 C e + 8 each), the previous coordinates and their inv entries read
    (12 each) and the previous rows inactive now written (C e each)."""
    from paper_2608_09388_amd.pipeline import SparseStack
    dev = torch.device("cuda:0")
    B, V, C = w.B, w.V, 128
    e = 2
    m_host = [w.mask.reshape(-1), synth.bernoulli_mask(B, V, float(w.mask.mean()),
                                                       synth._rng(11, 2)).reshape(-1)]
    md = [torch.from_numpy(np.ascontiguousarray(m.astype(np.uint8))).to(dev) for m in m_host]
    sets = []
    for m in md:
        coords = torch.empty((B * V, 2), dtype=torch.int32, device=dev)
        inv = torch.empty(B * V, dtype=torch.int32, device=dev)
        rp = torch.empty(B + 1, dtype=torch.int32, device=dev)
        nd = torch.empty(4, dtype=torch.int32, device=dev)
        ws = torch.empty(max(shc.compact_mask_workspace(B, V), 16), dtype=torch.uint8, device=dev)
        n = shc.compact_mask(m, B, V, coords, inv, rp, nd, ws)
        S = torch.randn((max(n, 1), C), device=dev).to(torch.bfloat16)
        sets.append((n, coords, inv, S))
    (na, ca, ia, Sa), (nb, cb, ib, Sb) = sets
    D = torch.zeros((B * V, C), dtype=torch.bfloat16, device=dev)
    ref = [torch.empty_like(D), torch.empty_like(D)]
    zf = shc.prepare_scatter(Sa, ia, ca, B, V, ref[0])
    shc.scatter(Sb, ib, cb, nb, B, V, ref[1], zero_fill=True)
    to_b = shc.prepare_scatter_update(Sb, ib, cb, ca, B, V, D)
    to_a = shc.prepare_scatter_update(Sa, ia, ca, cb, B, V, D)
    zf(na)
    shc.scatter(Sa, ia, ca, na, B, V, D, zero_fill=True)
    to_b(nb, na)
    torch.cuda.synchronize()
    same = bool(torch.equal(D, ref[1]))
    to_a(na, nb)
    torch.cuda.synchronize()
    same = same and bool(torch.equal(D, ref[0]))
    t_zf = _time_us(lambda: zf(na), torch, reps)
    t_pair = _time_us(lambda: (to_b(nb, na), to_a(na, nb)), torch, reps)
    torch.cuda.synchronize()
    same = same and bool(torch.equal(D, ref[0]))
    both = set(map(tuple, ca[:na].cpu().numpy().tolist())) & set(
        map(tuple, cb[:nb].cpu().numpy().tolist()))
    kept = len(both)
    upd_bytes = ((na + nb) * (2 * C * e + 8) + (na + nb) * 12
                 + (na - kept + nb - kept) * C * e) / 2
    zf_bytes = na * C * e + B * V * (4 + C * e)
    t_upd = t_pair / 2
    res = {"config": f"two Bernoulli masks of the density-sweep batch alternated "
                     f"(N'={na} and {nb}, {kept} rows in both), C={C} bf16",
           "update_equals_zero_fill": same,
           "zero_fill_scatter_us": round(t_zf, 2),
           "zero_fill_frac_hbm": round(zf_bytes / (t_zf * 1e-6) / 1e9 / HBM_PEAK_GBS, 4),
           "update_us": round(t_upd, 2),
           "update_algorithmic_bytes": int(upd_bytes),
           "update_frac_hbm": round(upd_bytes / (t_upd * 1e-6) / 1e9 / HBM_PEAK_GBS, 4)}
    del to_a, to_b, zf, D, ref, sets
    # the whole step, masks alternating, with each scatter
    for inc in (False, True):
        st = SparseStack(w, device="cuda:0", side_stream=True, incremental_scatter=inc)

        def feed(k, st=st):
            st.mask.copy_(md[k % 2])

        st.run(warmup, feed=feed)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        n_last = st.run(steps, feed=feed)
        torch.cuda.synchronize()
        ms = (time.perf_counter() - t0) * 1e3 / steps
        key = "step_ms_update" if inc else "step_ms_zero_fill"
        res[key] = round(ms, 4)
        res[key.replace("step_ms", "rows_per_s_per_layer")] = round(
            (na + nb) / 2 * len(w.layers) / (ms / 1e3), 1)
        del st
    res["steps"] = steps
    return res


def group_norm_measure(st, shc, torch, reps, G=32):
    """Sparse group normalization (Eqs. 7-9) of the conv layer's output rows,
    per body and channel group: back-to-back launches between HIP events on
    the stream it runs on, and its HBM fraction (one read and one write of
    every active value, plus the body offsets)."""
    n = st.n
    S = st.acts[-1]
    C = S.shape[-1]
    out = torch.empty_like(S)
    call = shc.prepare_segment_group_norm(S, st.row_ptr, st.B, G, out)
    for _ in range(3):
        call(n)
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    a.record()
    for _ in range(reps):
        call(n)
    b.record()
    torch.cuda.synchronize()
    us = a.elapsed_time(b) / reps * 1e3
    nbytes = 2 * n * C * S.element_size() + 4 * (st.B + 1)
    ach = nbytes / (us * 1e-6) / 1e9
    return {"config": f"N'={n} rows of the density-sweep conv output, C={C}, G={G}, "
                      f"{st.B} bodies", "launch_us": round(us, 2), "algorithmic_bytes": nbytes,
            "achieved": round(ach, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": round(ach / HBM_PEAK_GBS, 4)}


def backward_measure(st, w, shc, torch, reps):
    """Backward of the step's two layers (sparse linear + ReLU, then sparse
    conv + ReLU) on the density-sweep workload, with a seeded upstream
    gradient at the conv's output: the conv's input, weight and bias
    gradients, then the linear layer's from the conv's input gradient.  The
    transposed neighbour lists are built once per mesh, the transposed table
    and the slot pair lists once per active set (shared by every conv layer
    on it); each is timed on its own.  Prepared calls, back to back between
    HIP events.

    Roofline figure of the conv backward: algorithmic bytes (dY and the
    stored output Y read once, S and the input rows read once, the table,
    the row masks and the live transposed-table entries, dS and dW written
    once) over its time; flops 4 P C_in C_out for P present (row, slot)
    pairs (dW and dS each 2 P C_in C_out)."""
    n = st.n
    st.gather()                       # the step fuses it into the linear; the backward reads it
    K = w.K
    nbr_t, slot_of, Kt = shc.transpose_neighbors(st.nbr)
    table_t = torch.empty((Kt, n), dtype=torch.int32, device=st.device)
    row_slots = torch.empty(n, dtype=torch.int64, device=st.device)
    tt = shc.prepare_build_transposed_table(st.coords, st.inv, st.B, st.V, nbr_t, Kt, table_t,
                                            row_slots)
    tt(n)
    pairs = torch.empty((K * n, 2), dtype=torch.int32, device=st.device)
    pair_ptr = torch.empty(K + 1, dtype=torch.int32, device=st.device)
    sp = shc.prepare_build_slot_pairs(st.table, K, pairs, pair_ptr, n)
    sp(n)
    C0, C1, C2 = st.acts[0].shape[-1], st.acts[1].shape[-1], st.acts[2].shape[-1]
    g = torch.Generator(device=st.device).manual_seed(5)
    dY2 = torch.randn((n, C2), device=st.device, generator=g).to(st.dtype)
    dS1 = torch.empty((n, C1), dtype=st.dtype, device=st.device)
    dW1 = torch.empty(tuple(st.weights[1].shape), dtype=torch.float32, device=st.device)
    db1 = torch.empty(C2, dtype=torch.float32, device=st.device)
    dS0 = torch.empty((n, C0), dtype=st.dtype, device=st.device)
    dW0 = torch.empty(tuple(st.weights[0].shape), dtype=torch.float32, device=st.device)
    db0 = torch.empty(C1, dtype=torch.float32, device=st.device)
    conv = shc.prepare_sparse_neighbor_conv_backward(st.acts[1], st.table, table_t, row_slots,
                                                     slot_of, Kt, st.weights[1], st.acts[2], dY2,
                                                     dS1, dW1, db1, pairs=pairs,
                                                     pair_ptr=pair_ptr)
    lin = shc.prepare_sparse_linear_backward(st.acts[0], st.weights[0], st.acts[1], dS1, dS0,
                                             dW0, db0)
    t_tt = _time_us(lambda: tt(n), torch, reps)
    t_sp = _time_us(lambda: sp(n), torch, reps)
    t_conv = _time_us(lambda: conv(n), torch, reps)
    t_lin = _time_us(lambda: lin(n), torch, reps)
    t_both = _time_us(lambda: (conv(n), lin(n)), torch, reps)
    P = int((st.table.view(-1)[: K * n] >= 0).sum().item())
    e = st.weights[1].element_size()
    nbytes = (2 * n * C2 * e + n * C1 * e + K * C1 * C2 * e + 4 * K * n + 8 * n + 4 * P
              + n * C1 * e + 4 * K * C1 * C2 + 4 * C2)
    flops = 4.0 * P * C1 * C2
    ach = nbytes / (t_conv * 1e-6) / 1e9
    return {"config": f"{w.name}: N'={n}, K={K}, C={C1}, bf16, "
                      f"{Kt} virtual slots, {P} present (row, slot) pairs",
            "transposed_table_us": round(t_tt, 2), "slot_pairs_us": round(t_sp, 2),
            "conv_backward_us": round(t_conv, 2),
            "linear_backward_us": round(t_lin, 2), "both_layers_us": round(t_both, 2),
            "conv_algorithmic_bytes": nbytes, "conv_achieved": round(ach, 1),
            "peak": HBM_PEAK_GBS, "unit": "GB/s", "conv_frac": round(ach / HBM_PEAK_GBS, 4),
            "conv_tflops": round(flops / (t_conv * 1e-6) / 1e12, 1)}


def _time_us(fn, torch, reps):
    for _ in range(3):
        fn()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    a.record()
    for _ in range(reps):
        fn()
    b.record()
    torch.cuda.synchronize()
    return a.elapsed_time(b) / reps * 1e3


def gather_scatter_measure(shc, synth, torch, reps):
    """The row gather (S' of Eq. 2) and the zero-fill scatter on their own, on
    the masks of the full-mesh (B = 256, V = 10475, C = 64: the cap as written
    and its 5% variant, fp32 and bf16), density-sweep (B = 128, C = 128 bf16,
    5%) and sequence (2048 frames of V = 655, C = 256 bf16, Markov runs)
    workloads: HBM rates against the algorithmic bytes, 8 + 2 C e per active
    row for the gather and C e per active row + (4 + C e) per dense vertex for
    the scatter.  Features are N(0, 1) made on the device."""
    dev = torch.device("cuda:0")
    pts3, _ = synth.mesh("ellipsoid", 10475, 9, 3)
    cases = [("full mesh, cap y<-0.6", lambda: synth.cap_mask(pts3, 256, -0.6, 0.02, synth._rng(3, 1)), 64, "f32"),
             ("full mesh, 5% cap", lambda: synth.cap_mask(pts3, 256, -0.845, 0.02, synth._rng(3, 1)), 64, "f32"),
             ("full mesh, 5% cap", lambda: synth.cap_mask(pts3, 256, -0.845, 0.02, synth._rng(3, 1)), 64, "bf16"),
             ("density sweep 5%", lambda: synth.bernoulli_mask(128, 10475, 0.05, synth._rng(4, 1)), 128, "bf16"),
             ("sequences", lambda: synth.markov_mask(32, 64, 655, 0.10, 8.0, synth._rng(5, 1)), 256, "bf16")]
    out = []
    for name, mk, C, dt in cases:
        m = mk()
        B, V = m.shape
        td = torch.float32 if dt == "f32" else torch.bfloat16
        e = 4 if dt == "f32" else 2
        md = torch.from_numpy(np.ascontiguousarray(m.reshape(-1))).to(dev)
        coords = torch.empty((B * V, 2), dtype=torch.int32, device=dev)
        inv = torch.empty(B * V, dtype=torch.int32, device=dev)
        rp = torch.empty(B + 1, dtype=torch.int32, device=dev)
        nd = torch.empty(4, dtype=torch.int32, device=dev)
        ws = torch.empty(max(shc.compact_mask_workspace(B, V), 16), dtype=torch.uint8, device=dev)
        n = shc.compact_mask(md, B, V, coords, inv, rp, nd, ws)
        x = torch.randn((B * V, C), device=dev).to(td)
        S = torch.empty((max(n, 1), C), dtype=td, device=dev)
        D = torch.empty((B * V, C), dtype=td, device=dev)
        # prepared calls: one ctypes call per launch, so the host keeps ahead
        gather = shc.prepare_gather_rows(x, coords, B, V, S)
        scatter = shc.prepare_scatter(S, inv, coords, B, V, D)
        g_us = _time_us(lambda: gather(n), torch, reps)
        s_us = _time_us(lambda: scatter(n), torch, reps)
        g_b = n * (8 + 2 * C * e)
        s_b = n * C * e + B * V * (4 + C * e)
        out.append({"workload": name, "timing": "warm: back to back, inputs and part of the "
                                                 "output left in the caches by the launch before",
                    "B": B, "V": V, "C": C, "dtype": dt, "n_active": n,
                    "gather_us": round(g_us, 2),
                    "gather_frac_hbm": round(g_b / (g_us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4),
                    "scatter_us": round(s_us, 2),
                    "scatter_frac_hbm": round(s_b / (s_us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4)})
        del gather, scatter, x, S, D, coords, inv
    return out


def multi_mask_measure(st, w, shc, synth, torch, reps, kappa=3):
    """Several masks on the same input (kappa = 3 stacked as bodies k*B + b,
    each Bernoulli at the workload's density) and a mask drawn per element:
    HBM rates of the stacked gather, of the combination of the kappa dense
    outputs, of the per-element row activity and of the masked gather."""
    dev = st.device
    B, V, C = w.B, w.V, st.x.shape[-1]
    e = st.x.element_size()
    rng = np.random.default_rng(4242)
    masks = (rng.random((kappa * B, V)) < float(w.mask.mean())).astype(np.uint8)
    md = torch.from_numpy(masks.reshape(-1)).to(dev)
    Bs = kappa * B
    coords = torch.empty((Bs * V, 2), dtype=torch.int32, device=dev)
    inv = torch.empty(Bs * V, dtype=torch.int32, device=dev)
    rp = torch.empty(Bs + 1, dtype=torch.int32, device=dev)
    nd = torch.empty(4, dtype=torch.int32, device=dev)
    ws = torch.empty(max(shc.compact_mask_workspace(Bs, V), 16), dtype=torch.uint8, device=dev)
    n = shc.compact_mask(md, Bs, V, coords, inv, rp, nd, ws)
    S = torch.empty((n, C), dtype=st.x.dtype, device=dev)
    res = {"config": f"kappa={kappa} masks at p={float(w.mask.mean()):.3f} stacked as "
                     f"{Bs} bodies of V={V}, C={C}, N'={n}"}

    def rate(name, us, nbytes):
        ach = nbytes / (us * 1e-6) / 1e9
        res[name] = {"launch_us": round(us, 2), "algorithmic_bytes": int(nbytes),
                     "achieved": round(ach, 1), "unit": "GB/s",
                     "frac": round(ach / HBM_PEAK_GBS, 4)}

    us = _time_us(lambda: shc.gather_rows_stacked(st.x, coords, n, B, kappa, V, S), torch, reps)
    rate("gather_stacked", us, n * (8 + 2 * C * e))
    Y = torch.randn((Bs * V, C), device=dev).to(st.x.dtype)
    Dc = torch.empty((B * V, C), dtype=st.x.dtype, device=dev)
    us = _time_us(lambda: shc.combine_stacked(Y, kappa, B * V, Dc, "mean"), torch, reps)
    rate("combine_dense_mean", us, (kappa + 1) * B * V * C * e)
    del Y, Dc
    me = (torch.rand((B * V, C), device=dev) < 0.002).to(torch.uint8)
    m = torch.empty(B * V, dtype=torch.uint8, device=dev)
    us = _time_us(lambda: shc.row_mask_from_elements(me, B, V, m), torch, reps)
    rate("row_activity", us, B * V * (C + 1))
    n2 = shc.compact_mask(m, B, V, coords, inv, rp, nd, ws)
    S2 = torch.empty((n2, C), dtype=st.x.dtype, device=dev)
    us = _time_us(lambda: shc.gather_rows_masked(st.x, me, coords, n2, B, V, S2), torch, reps)
    rate("gather_masked", us, n2 * (8 + C + 2 * C * e))
    res["masked_rows"] = n2
    return res


def mask_scores_measure(w, shc, torch, reps, K=10, bodies=16):
    """Eq. 3 mask scores for K masks whose outputs are the dense per-vertex
    outputs of `bodies` bodies of the workload's mesh (N = bodies * V rows,
    C = 128, bf16): the whole call (Gram tiles, split reduction, scores and
    top-3), and the MFMA rate of its useful work, K(K+1)/2 Gram blocks of
    2 N C^2 flop each."""
    N, C = bodies * w.V, 128
    g = torch.Generator(device="cuda").manual_seed(7)
    Y = torch.randn((K, N, C), device="cuda", generator=g).to(torch.bfloat16)
    a_in = torch.zeros(K, dtype=torch.float64, device="cuda")
    a_out = torch.empty_like(a_in)
    top = torch.empty(3, dtype=torch.int32, device="cuda")
    ws = shc.mask_scores(Y, a_in, a_out, 3, top)
    us = _time_us(lambda: shc.mask_scores(Y, a_in, a_out, 3, top, None, ws), torch, reps)
    flops = K * (K + 1) / 2 * 2.0 * N * C * C
    ach = flops / (us * 1e-6) / 1e12
    return {"config": f"K={K} masks, N={N} rows ({bodies} bodies x V={w.V}), C={C}, bf16",
            "launch_us": round(us, 2), "useful_flops": flops, "achieved": round(ach, 1),
            "peak": BF16_MFMA_PEAK_TFLOPS, "unit": "TFLOP/s",
            "frac": round(ach / BF16_MFMA_PEAK_TFLOPS, 4), "bound": "mfma"}


def _time_each(fn, torch, reps, flush=None):
    """Durations (us) of `reps` launches of fn, each between its own pair of
    HIP events on the current stream; with `flush`, it runs before each
    launch (outside the events)."""
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(reps)]
    for _ in range(3):
        fn()
    torch.cuda.synchronize()
    for a, b in evs:
        if flush is not None:
            flush()
        a.record()
        fn()
        b.record()
    torch.cuda.synchronize()
    return np.array([a.elapsed_time(b) * 1e3 for a, b in evs])


def _pct(t):
    return {"p10": round(float(np.percentile(t, 10)), 2), "p50": round(float(np.median(t)), 2),
            "p90": round(float(np.percentile(t, 90)), 2), "reps": int(len(t))}


def cold_warm_measure(st, torch, reps=100):
    """The gather + linear layer, the conv and the zero-fill scatter of the
    step, each launched `reps` times on its own: warm (back to back, inputs
    left in the caches by the launch before) and cold (a 512 MiB write between
    launches evicts the 256 MiB Infinity Cache and the L2s), with p10 / p50 /
    p90 of the per-launch event times.  The flush reads its 512 MiB (a sum),
    so it leaves no dirty lines whose write-back would run during the next
    launch.  A per-launch event pair adds a few us of its own to short
    kernels, so the back-to-back averages of `per_kernel_us` stay the
    reference figures."""
    junk = torch.ones(512 * 1024 * 1024 // 4, dtype=torch.float32, device=st.device)
    acc = torch.zeros((), dtype=torch.float32, device=st.device)

    def flush():
        torch.sum(junk, dim=(0,), out=acc)

    lin = "gather+linear" if st.fused_gather else "linear"
    calls = {lin: lambda: st.layer(0), "conv": lambda: st.layer(1), "scatter": st.scatter,
             # reference: a plain write of the same dense output (PyTorch's fill)
             "fill_dense_output": lambda: st.dense_out.zero_()}
    out = {}
    for name, fn in calls.items():
        out[name] = {"warm": _pct(_time_each(fn, torch, reps)),
                     "cold": _pct(_time_each(fn, torch, reps, flush))}
    nb = st.dense_out.numel() * st.dense_out.element_size()
    out["fill_dense_output"]["bytes"] = nb
    out["fill_dense_output"]["cold_frac_hbm"] = round(
        nb / (out["fill_dense_output"]["cold"]["p50"] * 1e-6) / 1e9 / HBM_PEAK_GBS, 4)
    n = st.n
    sb = n * st.dense_out.shape[1] * st.dense_out.element_size() + st.B * st.V * (
        4 + st.dense_out.shape[1] * st.dense_out.element_size())
    out["scatter"]["cold_frac_hbm"] = round(sb / (out["scatter"]["cold"]["p50"] * 1e-6) / 1e9
                                            / HBM_PEAK_GBS, 4)
    del junk
    return out


def density_sweep(w0, shc, synth, torch, reps):
    """The density-sweep workload at every density it names (B = 128,
    V = 10475, K = 9, C = 128 bf16, i.i.d. Bernoulli(p)): the sparse linear
    layer (with the gather fused in) and the sparse conv, back to back on one
    stack per density, against the same layers at p = 1 (every vertex active:
    this library's dense run) and against PyTorch's dense layers (hipBLASLt
    matmul, an index_select per slot for the conv).  The crossover is the
    density where a sparse layer's time reaches its dense time (linear
    interpolation between sweep points)."""
    import copy
    from paper_2608_09388_amd.pipeline import SparseStack

    dens = [0.01, 0.05, 0.20, 0.50, 1.00]
    rows = []
    for p in dens:
        w = copy.copy(w0)
        w.mask = synth.bernoulli_mask(w0.B, w0.V, p, synth._rng(4, 1))
        st = SparseStack(w, device="cuda:0")
        n = st.compact()
        st.gather()
        st.layer(0)
        t_lin = _time_us(lambda: st.layer(0), torch, reps)
        t_conv = _time_us(lambda: st.layer(1), torch, reps)
        coords = st.coords[:n].cpu().numpy()
        inv = st.inv.cpu().numpy()
        cb, cf, a = algorithmic_conv(w, coords, inv, n, 2)
        lb = n * (8 + 2 * 128 * 2) + 128 * 128 * 2
        rows.append({"p": p, "n_active": n,
                     "linear_us": round(t_lin, 2), "conv_us": round(t_conv, 2),
                     "linear_rows_per_s": round(n / (t_lin * 1e-6), 1),
                     "conv_rows_per_s": round(n / (t_conv * 1e-6), 1),
                     "linear_frac_hbm": round(lb / (t_lin * 1e-6) / 1e9 / HBM_PEAK_GBS, 4),
                     "conv_frac_hbm": round(cb / (t_conv * 1e-6) / 1e9 / HBM_PEAK_GBS, 4),
                     "conv_useful_tflops": round(cf / (t_conv * 1e-6) / 1e12, 1),
                     "present_slot_fraction": round(a, 4)})
        if p == 1.0:
            # PyTorch's dense layers on the same all-rows input
            x = st.acts[1]
            Wl = st.weights[0]
            Wc = st.weights[1].reshape(-1, st.weights[1].shape[-1]).contiguous()
            nbr_flat = st.nbr.long().view(-1)
            BV = w.B * w.V
            t_lt = _time_us(lambda: torch.relu(st.x @ Wl), torch, 5)
            t_ct = _time_us(lambda: torch.relu(
                x.view(w.B, w.V, -1)[:, nbr_flat].reshape(BV, -1) @ Wc), torch, 3)
        del st
        torch.cuda.empty_cache()
    dense_lin, dense_conv = rows[-1]["linear_us"], rows[-1]["conv_us"]
    for r in rows:
        r["linear_speedup_vs_own_dense"] = round(dense_lin / r["linear_us"], 2)
        r["conv_speedup_vs_own_dense"] = round(dense_conv / r["conv_us"], 2)
        r["linear_speedup_vs_torch_dense"] = round(t_lt / r["linear_us"], 2)
        r["conv_speedup_vs_torch_dense"] = round(t_ct / r["conv_us"], 2)

    def crossover(key, dense):
        """Lowest density where the sparse layer takes as long as the dense
        one (interpolated), or None when it stays faster up to p < 1 (at
        p = 1 the sparse path is the dense run itself)."""
        prev = None
        for r in rows:
            if r["p"] < 1.0 and r[key] >= dense:
                if prev is None:
                    return r["p"]
                f = (dense - prev[key]) / (r[key] - prev[key])
                return round(prev["p"] + f * (r["p"] - prev["p"]), 3)
            prev = r
        return None

    return {"workload": "B=128, V=10475 ellipsoid, K=9, C=128->128 bf16, Bernoulli(p)",
            "points": rows, "dense_torch_linear_us": round(t_lt, 2),
            "dense_torch_conv_us": round(t_ct, 2),
            "crossover_vs_own_dense": {"linear": crossover("linear_us", dense_lin),
                                       "conv": crossover("conv_us", dense_conv)},
            "crossover_vs_torch_dense": {"linear": crossover("linear_us", t_lt),
                                         "conv": crossover("conv_us", t_ct)}}


def c3_layers(shc, synth, torch, reps):
    """The full-mesh workload's conv layer (B = 256, V = 10475, K = 9,
    C = 64 -> 64 + ReLU) in fp32 and bf16, with the cap mask as written and
    its 5% variant: rows/s, HBM fraction of the algorithmic bytes, and the
    useful MFMA rate against the dtype's peak (fp32 157.3, bf16 2500 TFLOP/s)."""
    from paper_2608_09388_amd.pipeline import SparseStack

    out = []
    for dt, five in (("f32", False), ("bf16", False), ("f32", True), ("bf16", True)):
        w = synth.workload_c3(dt, five_percent=five)
        st = SparseStack(w, device="cuda:0")
        n = st.compact()
        st.gather()
        t = _time_us(lambda: st.layer(0), torch, reps)
        e = 4 if dt == "f32" else 2
        coords = st.coords[:n].cpu().numpy()
        inv = st.inv.cpu().numpy()
        cb, cf, a = algorithmic_conv(w, coords, inv, n, e, layer=0)
        peak = 157.3 if dt == "f32" else BF16_MFMA_PEAK_TFLOPS
        out.append({"mask": "5% cap" if five else "cap y<-0.6", "dtype": dt, "n_active": n,
                    "conv_us": round(t, 2), "rows_per_s": round(n / (t * 1e-6), 1),
                    "algorithmic_bytes": int(cb),
                    "frac_hbm": round(cb / (t * 1e-6) / 1e9 / HBM_PEAK_GBS, 4),
                    "useful_tflops": round(cf / (t * 1e-6) / 1e12, 1),
                    "useful_frac_mfma": round(cf / (t * 1e-6) / 1e12 / peak, 4),
                    "present_slot_fraction": round(a, 4)})
        del st
        torch.cuda.empty_cache()
    return out


def dense_comparison(st, w, per_kernel_ms, torch, shc, synth):
    """Each sparse layer against the same layer run densely on all B*V rows:
    (i) this library's kernels with every vertex active, (ii) PyTorch-ROCm
    (hipBLASLt) matmul, with an index_select for the conv."""
    import copy
    from paper_2608_09388_amd.pipeline import SparseStack

    wd = copy.copy(w)
    wd.mask = np.ones_like(w.mask)
    sd = SparseStack(wd, device="cuda:0")
    sd.compact()
    sd.gather()

    def time_it(fn, reps=10):
        for _ in range(3):
            fn()
        s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        s.record()
        for _ in range(reps):
            fn()
        e.record()
        torch.cuda.synchronize()
        return s.elapsed_time(e) / reps

    lin_key = "gather+linear" if st.fused_gather else "linear"
    t_lin_own = time_it(lambda: sd.layer(0))
    t_conv_own = time_it(lambda: sd.layer(1))
    x = sd.acts[1]
    Wl = sd.weights[0]
    Wc = sd.weights[1].reshape(-1, sd.weights[1].shape[-1]).contiguous()
    nbr_flat = sd.nbr.long()
    BV = w.B * w.V

    def torch_linear():
        torch.relu(x @ Wl)

    def torch_conv():
        xg = x.view(w.B, w.V, -1)[:, nbr_flat.view(-1)].reshape(BV, -1)
        torch.relu(xg @ Wc)

    t_lin_t = time_it(torch_linear, 5)
    t_conv_t = time_it(torch_conv, 5)
    res = {
        "linear": {"sparse_us": round(per_kernel_ms[lin_key] * 1e3, 2),
                   "dense_own_kernel_us": round(t_lin_own * 1e3, 2),
                   "dense_torch_hipblaslt_us": round(t_lin_t * 1e3, 2),
                   "speedup_vs_own_dense": round(t_lin_own / per_kernel_ms[lin_key], 2),
                   "speedup_vs_torch_dense": round(t_lin_t / per_kernel_ms[lin_key], 2),
                   "sparse_layer": lin_key},
        "conv": {"sparse_us": round(per_kernel_ms["conv"] * 1e3, 2),
                 "dense_own_kernel_us": round(t_conv_own * 1e3, 2),
                 "dense_torch_gather_matmul_us": round(t_conv_t * 1e3, 2),
                 "speedup_vs_own_dense": round(t_conv_own / per_kernel_ms["conv"], 2),
                 "speedup_vs_torch_dense": round(t_conv_t / per_kernel_ms["conv"], 2)},
        "dense_rows": BV,
    }
    del sd
    torch.cuda.empty_cache()
    return res


if __name__ == "__main__":
    main()
