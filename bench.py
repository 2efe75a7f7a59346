#!/usr/bin/env python
"""Benchmark of GraphSAGE feature propagation (forward + backward) on MI355X.

One step is one pass of the whole hot path over one sampled subgraph:
per-subgraph preparation (transposed values of Algorithm 6, aggregation
plan), then for every layer the forward pass (aggregation, matrix-core
transforms, concat + ReLU) and, from the top layer down, the backward pass
(ReLU mask, transposed aggregation, weight and input gradients).  The top
layer's gradient is a fixed synthetic N(0,1) matrix standing in for the
classifier and loss.  All inputs are resident in HBM before timing starts.

Prints one JSON line: `value` is milliseconds per subgraph layer
(forward + backward, step time / layers), with the dominant kernel's
roofline and the CPU oracle timed on this host as a reference.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "ms per subgraph layer fwd+bwd; SpMM HBM GB/s and GEMM MFMA util vs peak"
PEAK_HBM_GBS = 8000.0
PEAK_TFLOPS = {"f32": 157.3, "bf16": 2516.6}
# fp32 GEMMs run by default as six bf16 piece products per fp32 product on
# the bf16 matrix cores: their ceiling is the bf16 peak over six
SPLIT_PRODUCTS = 6
PEAK_SPLIT = PEAK_TFLOPS["bf16"] / SPLIT_PRODUCTS


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def measured_traffic(workload: str, dtype: str) -> dict:
    """HBM bytes per launch from the committed rocprofv3 FETCH_SIZE /
    WRITE_SIZE summary, per kernel, only where the kernel's source file is
    unchanged since the counters were taken (else None)."""
    import glob
    import hashlib
    out = {}
    for path in glob.glob(os.path.join(ROOT, "profiles", "hbm_traffic_*.json")):
        try:
            d = json.load(open(path))
        except (OSError, ValueError):
            continue
        if d.get("workload") != workload or d.get("dtype") != dtype:
            continue
        for k, v in d.get("kernels", {}).items():
            src = os.path.join(ROOT, v["source"])
            ok = os.path.exists(src) and hashlib.sha256(
                open(src, "rb").read()).hexdigest() == v["source_sha256"]
            out[k] = v["bytes_per_launch"] if ok else None
    return out


def measured_mfma_util(workload: str, dtype: str) -> dict:
    """rocprofv3 MfmaUtil (percent) per GEMM kind from the committed counter
    summary, only where the kernel's source file is unchanged since."""
    import glob
    import hashlib
    out = {}
    for path in glob.glob(os.path.join(ROOT, "profiles", "mfma_util_*.json")):
        try:
            d = json.load(open(path))
        except (OSError, ValueError):
            continue
        if d.get("workload") != workload or d.get("dtype") != dtype:
            continue
        for k, v in d.get("kernels", {}).items():
            src = os.path.join(ROOT, v["source"])
            ok = os.path.exists(src) and hashlib.sha256(
                open(src, "rb").read()).hexdigest() == v["source_sha256"]
            out[k] = v["mfma_util_pct"] if ok else None
    return out


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default=None)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-bf16", action="store_true",
                    help="skip the native fp32 and the bf16 matrix-core variants")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="target CPU time of the oracle baseline sample")
    ap.add_argument("--skip-input-grad", action="store_true",
                    help="do not compute the first layer's input gradient")
    ap.add_argument("--fuse-masks", action="store_true",
                    help="layers above the first write their dX already masked "
                         "(the layer below skips its masking pass)")
    ap.add_argument("--no-graph", action="store_true",
                    help="skip the step replayed from a HIP graph")
    ap.add_argument("--no-floor", action="store_true",
                    help="skip the aggregation's gather floor (keeps a profile of the "
                         "step free of its standalone launches)")
    ap.add_argument("--no-probe", action="store_true",
                    help="skip the matrix cores' sustained-rate probe (gnn_mfma_rate_probe)")
    ap.add_argument("--no-rownorm", action="store_true",
                    help="skip the step with GNN_FLAG_ROW_NORMALIZED")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the other workloads (one line each in `configs`)")
    ap.add_argument("--config-steps", type=int, default=10,
                    help="timed steps per workload in `configs`")
    ap.add_argument("--no-variants", action="store_true",
                    help="skip the GCN and MixHop layer timings")
    ap.add_argument("--no-train", action="store_true",
                    help="skip the full training iteration timing")
    ap.add_argument("--no-pipeline", action="store_true",
                    help="skip the sampled-training pipeline timing (Kronecker graph)")
    ap.add_argument("--pipeline-scale", type=int, default=20,
                    help="log2 of the Kronecker full graph's node count")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="first run one plain device-to-device copy of MIB MiB "
                         "(reference point for hardware byte counters)")
    return ap.parse_args()


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU: the path runs one subgraph per GPU and "
              "has no multi-GPU leg (requested --gpus %d, WORLD_SIZE %d)"
              % (args.gpus, world), file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2010_03166_amd import gnnprop as G
    from paper_2010_03166_amd import runtime, synth

    G.lib()  # fail loudly if the HIP library is not built
    name = args.workload or synth.BENCH_WORKLOAD
    wl = synth.WORKLOADS[name]
    torch.cuda.set_device(0)
    log("workload", name)
    inp = synth.workload_inputs(wl)
    g, x, params, dy = inp["graph"], inp["x"], inp["params"], inp["dy"]
    stats = g.stats()
    log("graph", stats)

    if args.calibrate_copy:
        nbytes = args.calibrate_copy << 20
        src = torch.ones(nbytes // 4, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        log("calibration copy: %d bytes read, %d bytes written" % (nbytes, nbytes))
        del src, dst

    pad = 16
    dg = runtime.DeviceGraph(g)
    st = runtime.SageStack(dg, params, wl.f_in, pad=pad, fuse_masks=args.fuse_masks)
    ld_x = (wl.f_in + pad - 1) // pad * pad
    X = runtime.padded(torch.from_numpy(x).cuda(), ld_x)
    dY = torch.from_numpy(dy).cuda()
    want_dx_first = not args.skip_input_grad

    def step():
        dg.prepare()
        st.forward(X)
        st.backward(dY, want_dx_first=want_dx_first)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    # timed region: wall clock and stream events around exactly K steps
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    e0.record()
    for _ in range(args.steps):
        step()
    e1.record()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms_step = (t1 - t0) * 1e3 / args.steps
    ms_step_events = e0.elapsed_time(e1) / args.steps
    log("step %.4f ms (wall), %.4f ms (events)" % (ms_step, ms_step_events))

    # the same K steps again with every kernel bracketed by HIP events on the
    # stream it runs on
    G.gnn_timer_reset()
    G.gnn_timer_enable(True)
    torch.cuda.synchronize()
    t2 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    ms_step_timed = (time.perf_counter() - t2) * 1e3 / args.steps
    G.gnn_timer_enable(False)
    kernels = {}
    for kname in G.KERNELS:
        ms, launches, work = G.gnn_timer_read(kname)
        if launches:
            kernels[kname] = {"ms_per_step": ms / args.steps,
                              "launches_per_step": launches / args.steps,
                              "avg_launch_us": 1e3 * ms / launches, "work": work / launches}
    G.gnn_timer_reset()

    dtype = "f32"
    gemm_names = [k for k in kernels if k.startswith("gemm_") and k != "gemm_reduce"]
    for k in gemm_names:
        kernels[k]["tflops"] = kernels[k]["work"] / (kernels[k]["avg_launch_us"] * 1e6)
    if "spmm" in kernels:
        kernels["spmm"]["gbs"] = kernels["spmm"]["work"] / (kernels["spmm"]["avg_launch_us"] * 1e3)
    # the dominant kernel among those with an algorithmic work model
    cands = [k for k in kernels if k in gemm_names or k == "spmm"]
    dom = max(cands, key=lambda k: kernels[k]["ms_per_step"])
    if dom in gemm_names:
        ach = kernels[dom]["tflops"]
        roof = {"kernel": dom, "bound": "mfma", "achieved": round(ach, 2),
                "peak": round(PEAK_SPLIT, 1), "unit": "TFLOP/s",
                "frac": round(ach / PEAK_SPLIT, 4), "traffic": None,
                "peak_basis": "fp32 flops (2 M N K) against the bf16 matrix-core peak "
                              "%.1f TFLOP/s over the %d bf16 products each fp32 product "
                              "takes" % (PEAK_TFLOPS["bf16"], SPLIT_PRODUCTS),
                "frac_of_f32_mfma_peak": round(ach / PEAK_TFLOPS["f32"], 4),
                "flops_per_launch": kernels[dom]["work"],
                "avg_launch_us": round(kernels[dom]["avg_launch_us"], 2)}
    else:
        ach = kernels[dom].get("gbs", 0.0)
        roof = {"kernel": dom, "bound": "hbm", "achieved": round(ach, 1),
                "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": round(ach / PEAK_HBM_GBS, 4), "traffic": None,
                "bytes_per_launch": kernels[dom]["work"],
                "avg_launch_us": round(kernels[dom]["avg_launch_us"], 2)}
    roof_spmm = None
    if "spmm" in kernels:
        a = kernels["spmm"]["gbs"]
        roof_spmm = {"kernel": "spmm", "bound": "hbm", "achieved": round(a, 1),
                     "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": round(a / PEAK_HBM_GBS, 4),
                     "bytes_per_launch": kernels["spmm"]["work"],
                     "avg_launch_us": round(kernels["spmm"]["avg_launch_us"], 2)}

    # the streaming rate this GPU actually gives: a 512 MiB device-to-device
    # copy (reads plus writes), the "achievable" line beside the 8 TB/s peak
    copy_gbs = stream_copy_gbs(torch)
    if roof_spmm is not None:
        roof_spmm["copy_gbs"] = round(copy_gbs, 1)
        roof_spmm["frac_of_copy"] = round(roof_spmm["achieved"] / copy_gbs, 4)

    if roof_spmm is not None and not args.no_floor:
        roof_spmm.update(gather_floor(torch, G, dg, wl.hidden, kernels["spmm"]["work"]))

    traffic = measured_traffic(name, dtype)
    if traffic.get(dom) is not None:
        roof["traffic"] = traffic[dom]
        # the counters' bytes over the same launch time (HBM plus MALL)
        roof["traffic_gbs"] = round(traffic[dom] / (kernels[dom]["avg_launch_us"] * 1e3), 1)
    if roof_spmm is not None:
        roof_spmm["traffic"] = traffic.get("spmm")
        if traffic.get("spmm") is not None:
            roof_spmm["traffic_gbs"] = round(
                traffic["spmm"] / (kernels["spmm"]["avg_launch_us"] * 1e3), 1)
    if dom in gemm_names:
        roof["mfma_util_pct"] = measured_mfma_util(name, dtype).get(dom)
        if not args.no_probe:
            # what the bf16 matrix cores sustain on this GPU with nothing
            # but MFMAs in the loop, and the shader clock under that load
            pr = mfma_probe(torch, G, G.GNN_PROBE_MFMA_BF16)
            ceil = pr["tflops"] / SPLIT_PRODUCTS
            roof["mfma_probe"] = {"bf16_tflops": pr["tflops"], "shader_ghz": pr["shader_ghz"],
                                  "frac_of_bf16_peak": round(pr["tflops"] / PEAK_TFLOPS["bf16"], 4),
                                  "split_ceiling_tflops": round(ceil, 1),
                                  "frac_of_split_ceiling": round(ach / ceil, 4)}
            log("mfma probe: bf16 %.1f TFLOP/s at %.3f GHz; %s at %.3f of the split "
                "ceiling it gives" % (pr["tflops"], pr["shader_ghz"], dom, ach / ceil))

    out = {
        "metric": METRIC,
        "value": round(ms_step / wl.layers, 5),
        "unit": "ms",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 5),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": dtype,
        "gemm_products": "fp32 operands split exactly into bf16 hi + mid + lo, six "
                         "piece products (bf16x6) on the bf16 matrix cores, fp32 "
                         "accumulation; aggregation and all storage fp32",
        "data": "synthetic",
        "config": {"workload": name, "n": wl.n, "nnz": stats["nnz"],
                   "max_deg": stats["max_deg"], "f_in": wl.f_in,
                   "hidden_per_half": wl.hidden, "layers": wl.layers,
                   "graph": "%s mean %g gamma %g kmax %s" % (wl.graph, wl.mean_deg,
                                                             wl.gamma, wl.kmax),
                   "input_grad_first_layer": want_dx_first},
        "roofline": roof,
        "roofline_spmm": roof_spmm,
        "ms_per_step_events": round(ms_step_events, 5),
        "ms_per_step_with_kernel_timer": round(ms_step_timed, 5),
        "kernels": {k: {kk: (round(vv, 4) if isinstance(vv, float) else vv)
                        for kk, vv in v.items()} for k, v in kernels.items()},
    }

    # the same step replayed from a HIP graph: one host launch per step
    # instead of one per kernel, which is what bounds the small workloads
    if not args.no_graph:
        out["graph_step"] = bench_graph(torch, step, st, wl, args, want_dx_first)
        log("graph replay: %.4f ms per step" % out["graph_step"]["ms_per_step"])

    # the same step with the other GEMM arithmetic, reported alongside:
    # native fp32 MFMA products, and bf16-rounded operands
    if not args.no_bf16:
        out["f32_mfma_variant"] = bench_mode(
            G, runtime, torch, dg, params, wl, X, dY, args, want_dx_first, pad,
            G.GNN_FLAG_F32_MFMA, "fp32 products on v_mfma_f32_32x32x2_f32, fp32 throughout",
            PEAK_TFLOPS["f32"])
        log("f32 MFMA variant: %.4f ms per step" % out["f32_mfma_variant"]["ms_per_step"])
        vr = out["f32_mfma_variant"].get("roofline")
        if not args.no_probe and vr and vr.get("unit") == "TFLOP/s":
            pr = mfma_probe(torch, G, G.GNN_PROBE_MFMA_F32)
            vr["mfma_probe"] = {"f32_tflops": pr["tflops"], "shader_ghz": pr["shader_ghz"],
                                "frac_of_f32_peak": round(pr["tflops"] / PEAK_TFLOPS["f32"], 4),
                                "frac_of_probe": round(vr["achieved"] / pr["tflops"], 4)}
        out["bf16_variant"] = bench_mode(
            G, runtime, torch, dg, params, wl, X, dY, args, want_dx_first, pad,
            G.GNN_FLAG_BF16, "bf16 GEMM operands, f32 accumulation and aggregation",
            PEAK_TFLOPS["bf16"])
        log("bf16 variant: %.4f ms per step" % out["bf16_variant"]["ms_per_step"])

    # the same step with A_s = D^-1 A taken from the pattern alone
    # (GNN_FLAG_ROW_NORMALIZED: the aggregations read no value arrays)
    if not args.no_rownorm:
        out["row_normalized_variant"] = bench_mode(
            G, runtime, torch, dg, params, wl, X, dY, args, want_dx_first, pad,
            G.GNN_FLAG_ROW_NORMALIZED, "f32; A_s = D^-1 A from the row pointers "
            "(GNN_FLAG_ROW_NORMALIZED), split products", PEAK_SPLIT)
        log("row-normalized variant: %.4f ms per step" %
            out["row_normalized_variant"]["ms_per_step"])

    # the GCN and MixHop layers (Section 2.1) on the same subgraph with the
    # symmetric normalisation, one layer each, forward + backward with dX
    if not args.no_variants:
        out["variants"] = bench_variants(G, runtime, synth, torch, np, g, x, wl, args)

    # one whole training iteration of Algorithm 1 on the same subgraph
    if not args.no_train:
        out["train_iteration"] = bench_train(G, runtime, synth, torch, dg, X, params, wl,
                                             args, ms_step)

    # Algorithm 8 end to end: host sampler threads, induction on the GPU,
    # training, on the paper's synthetic Kronecker graph
    if not args.no_pipeline:
        out["pipeline"] = bench_pipeline(G, runtime, synth, torch, np, args)

    # every other workload of the benchmark set, the same step timed the
    # same way (fewer steps), with the bf16 variant beside the fp32 one for
    # the 300-feature workload
    if not args.no_configs:
        out["configs"] = bench_configs(G, runtime, synth, torch, np, name, args)

    if not args.no_cpu_baseline:
        from oracle import oracle as O
        import numpy as np  # noqa: F811
        reps, t_cpu = 0, 0.0
        while reps == 0 or (t_cpu < args.cpu_seconds and reps < 8):
            t = time.perf_counter()
            O.transpose_values(g)
            O.sage_stack(g, x, params, dy, want_dx_first=want_dx_first)
            t_cpu += time.perf_counter() - t
            reps += 1
        out["cpu_baseline"] = {
            "value": round(t_cpu * 1e3 / reps / wl.layers, 3), "unit": "ms",
            "cores": O.num_threads(), "kind": "oracle",
            "sample": "%d full step(s) of the same workload (Algorithm 6 + %d "
                      "layers forward + backward), double precision, plain loops"
                      % (reps, wl.layers),
            "cpu_model": cpu_model(),
            "gpu_speedup": None}
        out["cpu_baseline"]["gpu_speedup"] = round(out["cpu_baseline"]["value"] / out["value"], 1)
        log("cpu oracle %.1f ms/layer on %d threads" % (
            out["cpu_baseline"]["value"], out["cpu_baseline"]["cores"]))
        # the oracle's own parallel speedup: the same step on one thread, for
        # this workload and the 1,000-node one (results are the same for any
        # thread count)
        threads = O.num_threads()
        single = {}
        try:
            O.set_num_threads(1)
            for wname in (synth.TINY_WORKLOAD, name):
                w = synth.WORKLOADS[wname]
                d = inp if wname == name else synth.workload_inputs(w)
                t = time.perf_counter()
                O.transpose_values(d["graph"])
                O.sage_stack(d["graph"], d["x"], d["params"], d["dy"],
                             want_dx_first=want_dx_first)
                ms1 = (time.perf_counter() - t) * 1e3 / w.layers
                single[wname] = {"ms_per_layer_1_thread": round(ms1, 3)}
                log("cpu oracle, 1 thread, %s: %.1f ms/layer" % (wname, ms1))
        finally:
            O.set_num_threads(threads)
        single[name]["parallel_speedup"] = round(
            single[name]["ms_per_layer_1_thread"] / out["cpu_baseline"]["value"], 2)
        out["cpu_baseline"]["single_thread"] = single
    print(json.dumps(out), flush=True)


def bench_mode(G, runtime, torch, dg, params, wl, X, dY, args, want_dx_first, pad,
               flags, label, peak):
    """The benchmark step with other GEMM arithmetic (layer flags), timed the
    same way; the dominant GEMM's TFLOP/s against the given peak."""
    st = runtime.SageStack(dg, params, wl.f_in, pad=pad, flags=flags)

    def step():
        dg.prepare()
        st.forward(X)
        st.backward(dY, want_dx_first=want_dx_first)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / args.steps
    G.gnn_timer_reset()
    G.gnn_timer_enable(True)
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    G.gnn_timer_enable(False)
    kb = {}
    for kname in G.KERNELS:
        kms, launches, work = G.gnn_timer_read(kname)
        if launches:
            kb[kname] = {"ms_per_step": round(kms / args.steps, 4),
                         "avg_launch_us": round(1e3 * kms / launches, 2)}
            if kname.startswith("gemm_") and kname != "gemm_reduce":
                kb[kname]["tflops"] = round(work / launches / (1e6 * kb[kname]["avg_launch_us"]), 1)
            if kname == "spmm":
                kb[kname]["gbs"] = round(work / launches / (1e3 * kb[kname]["avg_launch_us"]), 1)
    G.gnn_timer_reset()
    gb = [k for k in kb if "tflops" in kb[k]]
    dom = max(gb, key=lambda k: kb[k]["ms_per_step"])
    return {"value": round(ms / wl.layers, 5), "unit": "ms", "ms_per_step": round(ms, 5),
            "dtype": label,
            "roofline": {"kernel": dom, "bound": "mfma", "achieved": kb[dom]["tflops"],
                         "peak": peak, "unit": "TFLOP/s",
                         "frac": round(kb[dom]["tflops"] / peak, 4)},
            "kernels": kb}


def time_stack(G, runtime, torch, dg, params, wl, X, dY, steps, warmup, flags):
    """ms per step (wall, K steps after W warm-up) of prep + the stack forward
    + backward with the first layer's dX, and the per-kernel event times of a
    second pass of K steps."""
    st = runtime.SageStack(dg, params, wl.f_in, pad=16, flags=flags)

    def step():
        dg.prepare()
        st.forward(X)
        st.backward(dY, want_dx_first=True)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / steps
    G.gnn_timer_reset()
    G.gnn_timer_enable(True)
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    G.gnn_timer_enable(False)
    kb = {}
    for kname in G.KERNELS:
        kms, launches, work = G.gnn_timer_read(kname)
        if launches:
            us = 1e3 * kms / launches
            kb[kname] = {"ms_per_step": round(kms / steps, 4), "avg_launch_us": round(us, 2)}
            if kname.startswith("gemm_") and kname != "gemm_reduce":
                kb[kname]["tflops"] = round(work / launches / (1e6 * us), 1)
            if kname == "spmm":
                kb[kname]["gbs"] = round(work / launches / (1e3 * us), 1)
    G.gnn_timer_reset()
    del st
    return ms, kb


def bench_configs(G, runtime, synth, torch, np, skip, args):
    """The other workloads (every configuration but the headline one): ms
    per layer and per step, the dominant kernel (largest time per step among
    the GEMMs and the aggregation) against its ceiling, and the aggregation's
    algorithmic GB/s; for the 300-feature workload also the bf16-product
    variant."""
    res = {}
    steps, warmup = max(2, args.config_steps), 2
    for name, wl in synth.WORKLOADS.items():
        if name == skip:
            continue
        inp = synth.workload_inputs(wl)
        g, x, params, dy = inp["graph"], inp["x"], inp["params"], inp["dy"]
        dg = runtime.DeviceGraph(g)
        ld_x = (wl.f_in + 15) // 16 * 16
        X = runtime.padded(torch.from_numpy(x).cuda(), ld_x)
        dY = torch.from_numpy(dy).cuda()
        modes = [("f32", 0, PEAK_SPLIT)]
        if name == "cl2.3-n8000-f300-h512-L3":
            modes.append(("bf16", G.GNN_FLAG_BF16, PEAK_TFLOPS["bf16"]))
        entry = {"n": wl.n, "nnz": int(g.nnz), "f_in": wl.f_in, "hidden_per_half": wl.hidden,
                 "layers": wl.layers}
        for label, flags, peak in modes:
            ms, kb = time_stack(G, runtime, torch, dg, params, wl, X, dY, steps, warmup,
                                flags)
            cands = [k for k in kb if "tflops" in kb[k] or k == "spmm"]
            dom = max(cands, key=lambda k: kb[k]["ms_per_step"])
            if dom == "spmm":
                roof = {"kernel": dom, "bound": "hbm", "achieved": kb[dom]["gbs"],
                        "peak": PEAK_HBM_GBS, "unit": "GB/s",
                        "frac": round(kb[dom]["gbs"] / PEAK_HBM_GBS, 4)}
            else:
                roof = {"kernel": dom, "bound": "mfma", "achieved": kb[dom]["tflops"],
                        "peak": round(peak, 1), "unit": "TFLOP/s",
                        "frac": round(kb[dom]["tflops"] / peak, 4)}
            e = {"ms_per_layer": round(ms / wl.layers, 5), "ms_per_step": round(ms, 5),
                 "dominant": roof,
                 "aggregation_gbs": kb.get("spmm", {}).get("gbs"),
                 "kernels": kb}
            if label == "f32":
                entry.update(e)
            else:
                entry["bf16_variant"] = e
            log("%s %s: %.4f ms/layer, dominant %s %.3f of its ceiling" % (
                name, label, ms / wl.layers, dom, roof["frac"]))
        res[name] = entry
        del dg, X, dY
        torch.cuda.empty_cache()
    return res


def bench_train(G, runtime, synth, torch, dg, X, params, wl, args, ms_prop):
    """ms per training iteration: preparation, the stack forward, classifier
    and loss (the workload's class count and loss), the backward pass from
    the classifier's input gradient, and an Adam update of every weight."""
    c = synth.classifier_inputs(wl)
    T = torch.from_numpy(c["targets"]).cuda()
    tr = runtime.Trainer(dg, params, wl.f_in, c["w_mlp"], wl.multilabel, "adam", lr=1e-3)

    def it():
        dg.prepare()
        tr.step(X, T)

    for _ in range(args.warmup):
        it()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        it()
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / args.steps
    G.gnn_timer_reset()
    G.gnn_timer_enable(True)
    for _ in range(args.steps):
        it()
    torch.cuda.synchronize()
    G.gnn_timer_enable(False)
    kern = {}
    for kname in G.KERNELS:
        kms, launches, _ = G.gnn_timer_read(kname)
        if launches:
            kern[kname] = {"ms_per_iteration": round(kms / args.steps, 4),
                           "launches": launches // args.steps}
    G.gnn_timer_reset()
    loss = float(tr.loss.item())
    log("train iteration: %.4f ms (loss %.4f after %d Adam steps)" % (ms, loss, tr.t))
    return {"ms_per_iteration": round(ms, 5),
            "head": "%d classes, %s" % (wl.classes, "sigmoid, multi-label"
                                         if wl.multilabel else "softmax"),
            "optimizer": "adam", "propagation_share": round(ms_prop / ms, 4),
            "loss_after": round(loss, 6), "kernels": kern}


def bench_pipeline(G, runtime, synth, torch, np, args):
    """ms per training iteration when every iteration draws a new subgraph:
    frontier sampling (m 1000, budget 8000, eta 2, clip 16) on host threads,
    induction and row gathers on the GPU, a 2-layer GraphSAGE (hidden 512
    per half) with a 2-class softmax head and Adam, on a Kronecker graph of
    2^scale nodes, mean degree 16, 50 features (the paper's synthetic
    graphs).  Reported overlapped (pool + preparation stream one subgraph
    ahead) and serial (sample, induce, train one after the other)."""
    scale, m, budget, eta, clip, f, C, hid = args.pipeline_scale, 1000, 8000, 2.0, 16, 50, 2, 512
    t0 = time.perf_counter()
    full = synth.kronecker_graph(scale, 16.0, 0)
    rng = np.random.default_rng(np.random.SeedSequence([8, scale]))
    X = rng.standard_normal((full.n, f)).astype(np.float32)
    Y = synth.labels(full.n, C, False, rng)
    log("kronecker graph 2^%d: %d entries, built in %.1f s" % (scale, full.nnz,
                                                              time.perf_counter() - t0))
    params = [synth.LayerParams(synth.glorot(f, hid, rng), synth.glorot(f, hid, rng)),
              synth.LayerParams(synth.glorot(2 * hid, hid, rng), synth.glorot(2 * hid, hid, rng))]
    w_mlp = synth.glorot(2 * hid, C, rng)
    dev = runtime.FullGraphDevice(full, X, Y)
    try:
        threads = min(16, len(os.sched_getaffinity(0)))
    except AttributeError:
        threads = min(16, os.cpu_count() or 1)
    # sampler alone, one thread
    t0 = time.perf_counter()
    ns = [len(G.gnn_frontier_sample(full, m, budget, eta, clip, 3, k)) for k in range(4)]
    samp_ms = (time.perf_counter() - t0) * 1e3 / 4
    res = {"graph": "kronecker 2^%d nodes, mean degree 16, initiator [[0.9, 0.5], [0.5, 0.1]]"
                    % scale,
           "model": "2 layers, hidden 512 per half, 50 features, 2 classes softmax, Adam",
           "sampler": {"m": m, "budget": budget, "eta": eta, "clip": clip,
                       "ms_per_subgraph_one_thread": round(samp_ms, 3),
                       "nodes_mean": round(float(np.mean(ns)), 1)},
           "threads": threads}
    iters, warm = args.steps, args.warmup
    # overlapped
    pool = G.gnn_sampler_pool(full, m, budget, eta, clip, 1, threads, 2 * threads)
    pipe = runtime.SubgraphPipeline(dev, pool, max_nodes=budget)
    tr = None
    nnz = []
    for k in range(warm + iters):
        if k == warm:
            torch.cuda.synchronize()
            t0 = time.perf_counter()
        dg, Xs, Ts, _ = pipe.next()
        nnz.append(dg.nnz)
        if tr is None:
            tr = runtime.Trainer(dg, params, f, w_mlp, False, "adam", lr=1e-3)
        else:
            tr.bind(dg)
        tr.step(Xs, Ts)
        pipe.release()
    torch.cuda.synchronize()
    res["ms_per_iteration_overlapped"] = round((time.perf_counter() - t0) * 1e3 / iters, 4)
    pool.close()
    res["subgraph_nnz_mean"] = int(np.mean(nnz))
    # serial: sample (one thread), induce (waits for the entry count), train
    tr = None
    for k in range(warm + iters):
        if k == warm:
            torch.cuda.synchronize()
            t0 = time.perf_counter()
        nodes = G.gnn_frontier_sample(full, m, budget, eta, clip, 1, k)
        dg, Xs, Ts = dev.induce(nodes)
        if tr is None:
            tr = runtime.Trainer(dg, params, f, w_mlp, False, "adam", lr=1e-3)
        else:
            tr.bind(dg)
        tr.step(Xs, Ts)
        torch.cuda.synchronize()
    res["ms_per_iteration_serial"] = round((time.perf_counter() - t0) * 1e3 / iters, 4)
    # GPU-side preparation alone (induction + gathers + plan + transposed values)
    G.gnn_timer_reset()
    G.gnn_timer_enable(True)
    for k in range(iters):
        dev.induce(G.gnn_frontier_sample(full, m, budget, eta, clip, 1, k))
    torch.cuda.synchronize()
    G.gnn_timer_enable(False)
    prep = {}
    for kname in ("induce", "gather", "plan", "transpose"):
        ms, launches, _ = G.gnn_timer_read(kname)
        if launches:
            prep[kname] = round(ms / iters, 4)
    G.gnn_timer_reset()
    res["gpu_prep_ms_per_subgraph"] = prep
    log("pipeline: %.3f ms/iteration overlapped, %.3f serial (sampler %.2f ms on one thread, "
        "%d threads)" % (res["ms_per_iteration_overlapped"], res["ms_per_iteration_serial"],
                         samp_ms, threads))
    del dev
    return res


def mfma_probe(torch, G, kind, reps=3):
    """The sustained rate of the matrix cores on this GPU: gnn_mfma_rate_probe
    (register-operand MFMAs only, 512-thread workgroups, two per CU as in
    the split-product GEMM), timed with events on the stream it runs on,
    median of `reps` launches after one warm-up; and the shader clock that
    its first wavefront counted (s_memtime cycles over 100 MHz ticks)."""
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    blocks = 2 * cus
    bf16 = kind == G.GNN_PROBE_MFMA_BF16
    iters = 2000 if bf16 else 1000
    flop = (32 * 32 * 16 * 2 if bf16 else 32 * 32 * 2 * 2) * 4.0 * iters * blocks * 8
    sink = torch.empty(blocks * 512, device="cuda")
    clocks = torch.zeros(2, dtype=torch.int64, device="cuda")
    G.gnn_mfma_rate_probe(kind, blocks, iters, sink, clocks)
    torch.cuda.synchronize()
    us, ghz = [], []
    for _ in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        G.gnn_mfma_rate_probe(kind, blocks, iters, sink, clocks)
        e1.record()
        torch.cuda.synchronize()
        us.append(1e3 * e0.elapsed_time(e1))
        cyc, ticks = (int(v) for v in clocks.cpu())
        ghz.append(0.1 * cyc / ticks if ticks > 0 else 0.0)
    us.sort()
    ghz.sort()
    del sink, clocks
    return {"tflops": round(flop / (us[len(us) // 2] * 1e6), 1),
            "shader_ghz": round(ghz[len(ghz) // 2], 3)}


def gather_floor(torch, G, dg, w, bytes_per_launch, reps=50):
    """The aggregation's gather order on this GPU without its row
    bookkeeping (gnn_spmm_gather_floor: same grid, slices, lane groups,
    entry order and loads, one sum per lane), timed beside gnn_spmm on the
    same graph and width with events on the stream both run on: the floor
    for this access pattern against which the aggregation is measured."""
    x = torch.randn(dg.n, w, device="cuda")
    out = torch.empty(dg.n, w, device="cuda")
    csr = dg.struct()

    def timed(fn):
        fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return 1e3 * e0.elapsed_time(e1) / reps

    us_floor = timed(lambda: G.gnn_spmm_gather_floor(csr, 0, w, x, w, out, w))
    us_spmm = timed(lambda: G.gnn_spmm(csr, 0, w, x, w, out, w, None))
    del x, out
    return {"gather_floor_us": round(us_floor, 2),
            "spmm_same_call_us": round(us_spmm, 2),
            "frac_of_gather_floor": round(us_floor / us_spmm, 4),
            "gather_floor_gbs": round(bytes_per_launch / (us_floor * 1e3), 1)}


def cpu_model() -> str:
    """The host CPU's model name (as /proc/cpuinfo gives it), or ""."""
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return ""


def stream_copy_gbs(torch, mib: int = 512, reps: int = 5) -> float:
    """GB/s (bytes read plus written) of a device-to-device copy."""
    src = torch.ones((mib << 20) // 4, device="cuda")
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        dst.copy_(src)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    del src, dst
    return 2.0 * (mib << 20) / (ms * 1e6)


def bench_graph(torch, step, st, wl, args, want_dx_first):
    """The propagation step captured once in a HIP graph and replayed; the
    first replay's outputs and gradients are compared bit for bit with those
    of the last eager step (every kernel is deterministic)."""
    outs = [L[k] for i, L in enumerate(st.layers) for k in ("Y", "dW_self", "dW_neigh", "dX")
            if k != "dX" or i > 0 or want_dx_first]
    ref = [o.clone() for o in outs]
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        step()  # warm-up outside the capture
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=s):
        step()
    for o in outs:
        o.fill_(float("nan"))
    graph.replay()
    torch.cuda.synchronize()
    same = all(torch.equal(a, b) for a, b in zip(ref, outs))
    for _ in range(args.warmup):
        graph.replay()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        graph.replay()
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / args.steps
    del graph
    return {"value": round(ms / wl.layers, 5), "unit": "ms", "ms_per_step": round(ms, 5),
            "matches_eager": bool(same)}


def bench_variants(G, runtime, synth, torch, np, g, x, wl, args):
    """ms per layer (forward + backward, first-layer shape) of a GCN layer
    (f_in -> h), a MixHop layer with K = 2 hops of h/2 columns each, and a
    GAT layer (f_in -> h, attention slope 0.2)."""
    gs = synth.sym_normalized(g)
    dg = runtime.DeviceGraph(gs)
    dg.prepare()
    c = dg.struct()
    f_in, h, n = wl.f_in, wl.hidden, g.n
    pad = 16
    rup = lambda v: (v + pad - 1) // pad * pad
    rng = np.random.default_rng(5)
    X = runtime.padded(torch.from_numpy(x).cuda(), rup(f_in))
    res = {}

    def buf(nb):
        return torch.empty(max(int(nb), 256), dtype=torch.uint8, device="cuda")

    def timed(fn):
        for _ in range(args.warmup):
            fn()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(args.steps):
            fn()
        torch.cuda.synchronize()
        ms = (time.perf_counter() - t0) * 1e3 / args.steps
        G.gnn_timer_reset()
        G.gnn_timer_enable(True)
        for _ in range(args.steps):
            fn()
        torch.cuda.synchronize()
        G.gnn_timer_enable(False)
        kern = {}
        for kname in G.KERNELS:
            kms, launches, work = G.gnn_timer_read(kname)
            if launches:
                kern[kname] = {"ms_per_layer": round(kms / args.steps, 4),
                               "launches": launches // args.steps}
                if kname.startswith("gemm_") and kname != "gemm_reduce":
                    kern[kname]["tflops"] = round(work / kms / 1e9, 1)
        G.gnn_timer_reset()
        return ms, kern

    # GCN: Y = ReLU(A_hat X W)
    W = torch.from_numpy(synth.glorot(f_in, h, rng)).cuda()
    lay = G.make_layer(f_in, h, X.stride(0), rup(h), X.stride(0), 0, 0)
    Y = torch.empty((n, rup(h)), device="cuda")[:, :h]
    dY = torch.from_numpy(rng.standard_normal((n, h)).astype(np.float32)).cuda()
    dYp = runtime.padded(dY, rup(h))
    dX = torch.empty((n, rup(f_in)), device="cuda")[:, :f_in]
    dW = torch.empty((f_in, h), device="cuda")
    saved, ws = buf(G.gnn_gcn_saved_bytes(c, lay)), buf(G.gnn_gcn_workspace_bytes(c, lay))

    def gcn():
        G.gnn_gcn_fwd(c, lay, X, W, None, Y, saved, ws)
        G.gnn_gcn_bwd(c, lay, X, W, Y, dYp, saved, dX, dW, None, ws)

    ms, kern = timed(gcn)
    res["gcn"] = {"ms_per_layer": round(ms, 5), "shape": "%d -> %d, order %d" % (
        f_in, h, G.gnn_choose_order(f_in, h)), "kernels": kern}
    log("gcn layer: %.4f ms" % ms)
    # MixHop, K = 2 hops of h/2 columns: Y = ReLU(X W_0 || A X W_1 || A^2 X W_2)
    K, hk = 2, h // 2
    wy = (K + 1) * hk
    Wm = torch.from_numpy(synth.glorot(f_in, wy, rng)).cuda()
    laym = G.make_layer(f_in, hk, X.stride(0), rup(wy), X.stride(0), 0, 0)
    Ym = torch.empty((n, rup(wy)), device="cuda")[:, :wy]
    dYm = runtime.padded(torch.from_numpy(rng.standard_normal((n, wy)).astype(np.float32)).cuda(),
                         rup(wy))
    dWm = torch.empty((f_in, wy), device="cuda")
    savedm = buf(G.gnn_mixhop_saved_bytes(c, laym, K))
    wsm = buf(G.gnn_mixhop_workspace_bytes(c, laym, K))

    def mixhop():
        G.gnn_mixhop_fwd(c, laym, K, X, Wm, None, Ym, savedm, wsm)
        G.gnn_mixhop_bwd(c, laym, K, X, Wm, Ym, dYm, savedm, dX, dWm, None, wsm)

    ms, kern = timed(mixhop)
    res["mixhop_k2"] = {"ms_per_layer": round(ms, 5),
                        "shape": "%d -> 3 x %d" % (f_in, hk), "kernels": kern}
    log("mixhop layer: %.4f ms" % ms)
    # GAT: Y = ReLU(A_att X W), attention on the stored entries (row-normalised
    # pattern of the same subgraph; its values are not used)
    dgs = runtime.DeviceGraph(g)
    dgs.prepare()
    cg = dgs.struct()
    a = torch.from_numpy((rng.standard_normal(2 * h) / np.sqrt(h)).astype(np.float32)).cuda()
    layg = G.make_layer(f_in, h, X.stride(0), rup(h), X.stride(0), 0, 0)
    savedg, wsg = buf(G.gnn_gat_saved_bytes(cg, layg)), buf(G.gnn_gat_workspace_bytes(cg, layg))
    da = torch.empty(2 * h, device="cuda")

    def gat():
        G.gnn_gat_fwd(cg, layg, X, W, a, 0.2, Y, None, savedg, wsg)
        G.gnn_gat_bwd(cg, layg, X, W, a, 0.2, Y, dYp, savedg, dX, dW, da, wsg)

    ms, kern = timed(gat)
    res["gat"] = {"ms_per_layer": round(ms, 5), "shape": "%d -> %d" % (f_in, h),
                  "kernels": kern}
    log("gat layer: %.4f ms" % ms)
    return res


if __name__ == "__main__":
    main()
