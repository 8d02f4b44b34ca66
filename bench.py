"""Benchmark: training images/s and HBM bytes per step of DenseNet-121 dense
block 1 + transition (N=64, 56x56, bf16 operands, fp32 BN statistics), BN
fission/fusion path vs the unfused path, on one MI355X.

A step is one forward + backward pass of the whole block (six composite
layers + transition) over one batch of synthetic inputs already resident in
HBM.  Each variant's step is captured once in a HIP graph and replayed.
Variants: fused (BN fission/fusion + inter-composite-layer fusion: the
headline value), fused_no_icf (fission/fusion inside composite layers only)
and unfused (the reference layer chain).

Prints one JSON line (rank 0).  Options: --gpus (1 only), --steps, --warmup,
--workload {dense_block,bottleneck,single_layer,resnet_stack}, --no-graph,
--no-cpu-baseline, --profile-only (steps only, for rocprofv3 runs).
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

WORKLOADS = {
    "dense_block": ("DenseBlock", "dense_block", dict(n=64)),
    "bottleneck": ("Bottleneck", "bottleneck", dict(n=32)),
    "single_layer": ("SingleLayer", "single_layer", dict()),
    "resnet_stack": ("ResNetStack", "resnet_stack", dict(n=128)),
}


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="dense_block", choices=sorted(WORKLOADS))
    ap.add_argument("--no-graph", action="store_true")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--profile-only", action="store_true")
    ap.add_argument("--only", choices=["fused", "fused_no_icf", "unfused"], default=None)
    return ap.parse_args()


def build_workloads(args, torch):
    from paper_1807_01702_amd import synth
    from paper_1807_01702_amd import workloads as W
    cls, recipe, kw = WORKLOADS[args.workload]
    data = getattr(synth, recipe)(seed=0, **kw)
    variants = [("fused", dict(fused=True)), ("unfused", dict(fused=False))]
    if args.workload == "dense_block":          # fused = BNFF + inter-composite-layer fusion; BNFF alone beside it
        variants.insert(1, ("fused_no_icf", dict(fused=True, icf=False)))
    out = {}
    for name, kw in variants:
        if args.only and args.only != name:
            continue
        out[name] = getattr(W, cls)(data, **kw)
    return data, out


def timed_steps(torch, wl, steps, warmup, use_graph):
    for _ in range(warmup):
        wl.step()
    torch.cuda.synchronize()
    graph = None
    if use_graph:
        s = torch.cuda.Stream()
        s.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(s):
            wl.step()                    # first call on this stream outside capture
            torch.cuda.synchronize()
            graph = torch.cuda.CUDAGraph()
            with torch.cuda.graph(graph, stream=s):
                wl.step()
        torch.cuda.current_stream().wait_stream(s)
        torch.cuda.synchronize()
        for _ in range(2):
            graph.replay()
        torch.cuda.synchronize()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    start.record()
    for _ in range(steps):
        if graph is not None:
            graph.replay()
        else:
            wl.step()
    end.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    return start.elapsed_time(end) / steps, wall, graph


PEAK_HBM_GBS = 8000.0          # MI355X HBM3E
PEAK_MFMA_TFS = {"bf16": 2500.0, "f32": 157.3}


def traced_kernels(torch, wl, steps):
    """Per-kernel totals over `steps` eager steps, each launch bracketed by
    HIP events on its own stream inside the library."""
    from paper_1807_01702_amd import bnr as B
    wl.step()
    torch.cuda.synchronize()
    B.bnr_trace_begin(0xF, 200000)
    for _ in range(steps):
        wl.step()
    torch.cuda.synchronize()
    recs = B.bnr_trace_end(200000)
    agg = {}
    for name, ms, by, fl in recs:
        a = agg.setdefault(name, [0, 0.0, 0.0, 0.0])
        a[0] += 1
        a[1] += ms
        a[2] += by
        a[3] += fl
    out = {}
    for name, (n, ms, by, fl) in agg.items():
        out[name] = dict(launches_per_step=n / steps, ms_per_step=ms / steps, avg_launch_us=1e3 * ms / n,
                         algorithmic_bytes_per_launch=by / n, flops_per_launch=fl / n,
                         achieved_GBps=by / (ms * 1e-3) / 1e9 if ms > 0 else None)
    return out


def roofline(kernels, dtype):
    name = max(kernels, key=lambda k: kernels[k]["ms_per_step"])
    k = kernels[name]
    t = k["avg_launch_us"] * 1e-6
    bytes_t = k["algorithmic_bytes_per_launch"] / (PEAK_HBM_GBS * 1e9)
    flops_t = k["flops_per_launch"] / (PEAK_MFMA_TFS[dtype] * 1e12)
    if flops_t > bytes_t:
        ach = k["flops_per_launch"] / t / 1e12
        return dict(bound="mfma", achieved=ach, peak=PEAK_MFMA_TFS[dtype], unit="TFLOP/s",
                    frac=ach / PEAK_MFMA_TFS[dtype], traffic=None, kernel=name,
                    avg_launch_us=k["avg_launch_us"], flops_per_launch=k["flops_per_launch"])
    ach = k["algorithmic_bytes_per_launch"] / t / 1e9
    return dict(bound="hbm", achieved=ach, peak=PEAK_HBM_GBS, unit="GB/s", frac=ach / PEAK_HBM_GBS, traffic=None,
                kernel=name, avg_launch_us=k["avg_launch_us"],
                algorithmic_bytes_per_launch=k["algorithmic_bytes_per_launch"])


def cpu_baseline(args):
    """The fp64 oracle, as it stands, on a bounded sample of the same workload."""
    import numpy as np
    from oracle import compose as OC
    from paper_1807_01702_amd import synth
    threads = int(os.environ.get("OMP_NUM_THREADS", "0")) or len(os.sched_getaffinity(0))
    os.environ.setdefault("OMP_NUM_THREADS", str(threads))
    rnd = OC.storage(True)
    if args.workload == "dense_block":
        n = 64
        d = synth.dense_block(seed=0, n=n)
        t0 = time.perf_counter()
        _, c = OC.block_fwd(d["x"], d["cpls"], d["trans"], d["eps"], rnd, d["c_total"])
        OC.block_bwd(c, d["dpool"].astype(np.float64), rnd)
    elif args.workload == "bottleneck":
        n = 32
        d = synth.bottleneck(seed=0, n=n)
        t0 = time.perf_counter()
        _, c = OC.bottleneck_fwd(d["x"], d["p"]["w2"].shape[3], d["p"], d["eps"], rnd)
        OC.bottleneck_bwd(c, d["dy"].astype(np.float64), rnd)
    elif args.workload == "resnet_stack":
        n = 4                     # bounded sample: the stack at batch 4 (per-image cost is batch independent)
        d = synth.resnet_stack(seed=0, n=n)
        t0 = time.perf_counter()
        X, cs = d["x"], []
        for p in d["blocks"]:
            X, c = OC.resnet_block_fwd(X, p, d["eps"], rnd)
            cs.append(c)
        g = d["dy"].astype(np.float64)
        for c in reversed(cs):
            g, _ = OC.resnet_block_bwd(c, g, rnd)
    else:
        d = synth.single_layer(seed=0)
        n = d["x"].shape[0]
        rnd = OC.storage(False)
        t0 = time.perf_counter()
        c = OC.unit_fwd(d["x"], d["gamma"], d["beta"], d["w"], d["eps"], rnd)
        OC.unit_bwd(c, d["dy"].astype(np.float64), rnd)
    dt = time.perf_counter() - t0
    return {"value": n / dt, "unit": "images/s", "cores": threads, "kind": "oracle",
            "sample": "one %s training step (fwd+bwd) at batch %d, fp64 oracle with the configuration's storage "
                      "model; %.1f s on %d threads" % (args.workload, n, dt, threads)}


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py measures one GPU: this build has no multi-GPU path (run with --gpus 1)", file=sys.stderr)
        sys.exit(2)
    import torch
    from paper_1807_01702_amd import bytes_model
    torch.cuda.set_device(0)
    data, wls = build_workloads(args, torch)
    res = {}
    for name, wl in wls.items():
        ms, wall, _ = timed_steps(torch, wl, args.steps, args.warmup, not args.no_graph)
        res[name] = dict(ms=ms, wall=wall, images=wl.images)
    if args.profile_only:
        print(json.dumps({k: v["ms"] for k, v in res.items()}))
        return
    dtype = "bf16" if data.get("bf16") else "f32"
    kernels = traced_kernels(torch, wls["fused"], args.steps) if "fused" in wls else None
    fused = res.get("fused")
    unf = res.get("unfused")
    noicf = res.get("fused_no_icf")
    model = bytes_model.for_workload(args.workload, data)
    line = {
        "metric": "training images/sec + HBM bytes/step, DenseNet-121 block (fused vs unfused)",
        "value": fused["images"] / (fused["ms"] / 1e3) if fused else None,
        "unit": "images/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": fused["ms"] if fused else None,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": dtype,
        "data": "synthetic (seeded N(0,1) activations and gradients, He-normal weights)",
        "config": {"workload": {"dense_block": "DenseNet-121 dense block 1 (6 composite layers, growth 32, width "
                                               "128, 64->256 ch) + transition BN-ReLU-CONV1x1 256->128 + avgpool2",
                                "bottleneck": "DenseNet-121 bottleneck layer 256->128->32 + concat",
                                "single_layer": "BN-ReLU-CONV1x1 64->32",
                                "resnet_stack": "ResNet-50 conv2_x: 3 bottleneck blocks 256->64->64->256 with "
                                                "identity shortcuts"}[args.workload],
                   "global_batch": fused["images"] if fused else unf["images"], "image_hw": 56,
                   "graph": not args.no_graph},
        "unfused": {"images_per_s": unf["images"] / (unf["ms"] / 1e3), "ms_per_step": unf["ms"]} if unf else None,
        "fused_no_icf": ({"images_per_s": noicf["images"] / (noicf["ms"] / 1e3), "ms_per_step": noicf["ms"],
                          "algorithmic_bytes": model.get("fused_no_icf")} if noicf else None),
        "speedup_vs_unfused": (unf["ms"] / fused["ms"]) if (fused and unf) else None,
        "hbm_bytes_per_step": {"algorithmic_fused": model["fused"], "algorithmic_unfused": model["unfused"]},
        "roofline": roofline(kernels, dtype) if kernels else None,
        "kernels": kernels,
        "cpu_baseline": None if args.no_cpu_baseline else cpu_baseline(args),
    }
    print(json.dumps(line))


if __name__ == "__main__":
    main()
