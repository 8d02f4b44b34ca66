"""Benchmark: training images/s and HBM bytes per step of DenseNet-121 dense
block 1 + transition (N=64, 56x56, bf16 operands, fp32 BN statistics), BN
fission/fusion path vs the unfused path, on one MI355X.

A step is one forward + backward pass of the whole block (six composite
layers + transition) over one batch of synthetic inputs already resident in
HBM.  Each variant's step is captured once in a HIP graph and replayed.
Variants: fused (BN fission/fusion + inter-composite-layer fusion: the
headline value), fused_no_icf (fission/fusion inside composite layers only),
fused_o2 (that, with the paper's stored O2' sweep: the backward reads the
stored BN+ReLU outputs instead of recomputing them) and unfused (the
reference layer chain).

Prints one JSON line (rank 0).  Options: --gpus (1 only), --steps, --warmup,
--workload {dense_block,bottleneck,single_layer,resnet_stack,densenet121}, --no-graph,
--no-cpu-baseline, --profile-only (steps only, for rocprofv3 runs),
--calib-copy-mb M (with --profile-only: one bnr_hbm_copy of M MiB after the
steps, the byte-counter calibration reference), --only VARIANT, --no-ablation
(skip the unfused_rcf / unfused_rcf_mvf endpoints).

Counter summaries (no GPU needed): --summarize-pmc (per-class bytes of the
dominant-kernel roofline), --summarize-step-bytes FETCH_DIR WRITE_DIR (HBM bytes
per step of a profile-only run), --summarize-mfma PMC_DIR (matrix-core rate and
busy fraction per kernel class), --summarize-lds PMC_DIR (LDS instructions and
bank-conflict cycles per kernel class), --summarize-trace (rocprofv3 --stats tables).

HBM traffic of the dominant kernel (`roofline.traffic`): two rocprofv3
counter runs of the profile-only command, one with FETCH_SIZE and one with
WRITE_SIZE, are summarised by `python bench.py --summarize-pmc FETCH_DIR
WRITE_DIR --calib-copy-mb M` into profiles/hbm_traffic_<workload>.json: per kernel class the
counter bytes per launch, each scaled by expected / counted bytes of the
calibration copy, and the SHA-256 of the sources the class is built from.
The bench line reports that figure only while those sources are unchanged.
"""
import argparse
import csv
import glob
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

WORKLOADS = {
    "dense_block": ("DenseBlock", "dense_block", dict(n=64)),
    "bottleneck": ("Bottleneck", "bottleneck", dict(n=32)),
    "single_layer": ("SingleLayer", "single_layer", dict()),
    "resnet_stack": ("ResNetStack", "resnet_stack", dict(n=128)),
    "densenet121": ("DenseNet", "densenet", dict(n=128)),
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
    ap.add_argument("--only", choices=["fused", "fused_no_icf", "fused_o2", "fused_overlap", "fused_robust", "unfused",
                                       "unfused_rcf",
                                       "unfused_rcf_mvf"],
                    default=None)
    ap.add_argument("--no-ablation", action="store_true")
    ap.add_argument("--flush-mb", type=int, default=512,
                    help="MiB copied before every library call in the cold-cache trace (0: no cold-cache trace)")
    ap.add_argument("--bn-passes", type=int, default=0, metavar="MB",
                    help="time the standalone BN sweeps on tensors of about MB megabytes and exit")
    ap.add_argument("--summarize-step-bytes", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"), default=None)
    ap.add_argument("--summarize-ablation", metavar="RUN_DIR", default=None,
                    help="RUN_DIR/sb_f_V, RUN_DIR/sb_w_V of each variant V (profile-only runs, --steps 2 --warmup 1) "
                         "-> profiles/hbm_bytes_per_step_<workload>.json and a markdown table (with --bench-json)")
    ap.add_argument("--summarize-mfma", metavar="PMC_DIR", default=None)
    ap.add_argument("--summarize-lds", metavar="PMC_DIR", default=None)
    ap.add_argument("--calib-copy-mb", type=int, default=0)
    ap.add_argument("--summarize-pmc", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"), default=None)
    ap.add_argument("--summarize-trace", nargs=2, metavar=("KERNEL_STATS_CSV", "STEPS"), default=None)
    ap.add_argument("--bench-json", default=None)
    ap.add_argument("--summarize-bench", metavar="BENCH_JSON", default=None,
                    help="markdown: the bench line's figures, per-class event timings, warm and cold cache")
    return ap.parse_args()


def build_workloads(args, torch):
    from paper_1807_01702_amd import synth
    from paper_1807_01702_amd import workloads as W
    cls, recipe, kw = WORKLOADS[args.workload]
    data = getattr(synth, recipe)(seed=0, **kw)
    variants = [("fused", dict(fused=True)), ("unfused", dict(fused=False))]
    if args.workload == "dense_block":          # fused = BNFF + inter-composite-layer fusion; BNFF alone beside it
        variants.insert(1, ("fused_no_icf", dict(fused=True, icf=False)))
        # the same fused step with the weight gradients on a side stream
        variants.insert(2, ("fused_overlap", dict(fused=True, overlap=True)))
        # the same fused step with robust one-sweep statistics (sums around the running mean)
        variants.insert(3, ("fused_robust", dict(fused=True, robust=True)))
        # BNFF with the paper's stored O2' sweep (the backward reads relu(bn(x)) instead of recomputing it)
        variants.insert(2, ("fused_o2", dict(fused=True, icf=False, o2=True)))
    if args.workload in ("dense_block", "resnet_stack", "densenet121") and not args.no_ablation:
        # the paper's intermediate endpoints (Sec. 5): ReLU-CONV fusion, then + mean/variance fusion
        from paper_1807_01702_amd import bnr as B
        variants += [("unfused_rcf", dict(fused=False, ref_mode=B.MODE_RCF)),
                     ("unfused_rcf_mvf", dict(fused=False, ref_mode=B.MODE_RCF_MVF))]
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


def traced_kernels(torch, wl, steps, flush_mb=0):
    """Per-kernel totals over `steps` eager steps, each launch bracketed by
    HIP events on its own stream inside the library.  flush_mb > 0: before
    every library call of the step a copy of flush_mb MiB (read and written)
    evicts the L2 caches and the Infinity Cache (256 MB), so every kernel
    starts cold; the copies themselves are not counted."""
    from paper_1807_01702_amd import bnr as B
    wl.step()
    torch.cuda.synchronize()
    saved = {}
    if flush_mb > 0:
        n = flush_mb * 1024 * 1024 // 4
        fsrc = torch.ones(n, dtype=torch.float32, device="cuda")
        fdst = torch.empty_like(fsrc)
        copy = B.bnr_hbm_copy

        def cold(f):
            def g(*a, **k):
                copy(fsrc, fdst)
                return f(*a, **k)
            return g
        for name in dir(B):
            if name.startswith("bnr_") and name not in ("bnr_hbm_copy", "bnr_trace_begin", "bnr_trace_end") and \
                    callable(getattr(B, name)) and not name.endswith("_size"):
                saved[name] = getattr(B, name)
                setattr(B, name, cold(saved[name]))
    try:
        B.bnr_trace_begin(0xF, 200000)
        for _ in range(steps):
            wl.step()
        torch.cuda.synchronize()
        recs = B.bnr_trace_end(200000)
    finally:
        for name, f in saved.items():
            setattr(B, name, f)
    agg = {}
    for name, ms, by, fl in recs:
        if flush_mb > 0 and name == "copy":
            continue
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


def roofline(kernels, dtype, workload):
    name = max(kernels, key=lambda k: kernels[k]["ms_per_step"])
    traffic = traffic_for(workload, name)
    k = kernels[name]
    t = k["avg_launch_us"] * 1e-6
    bytes_t = k["algorithmic_bytes_per_launch"] / (PEAK_HBM_GBS * 1e9)
    flops_t = k["flops_per_launch"] / (PEAK_MFMA_TFS[dtype] * 1e12)
    if flops_t > bytes_t:
        ach = k["flops_per_launch"] / t / 1e12
        return dict(bound="mfma", achieved=ach, peak=PEAK_MFMA_TFS[dtype], unit="TFLOP/s",
                    frac=ach / PEAK_MFMA_TFS[dtype], traffic=traffic, kernel=name,
                    avg_launch_us=k["avg_launch_us"], flops_per_launch=k["flops_per_launch"])
    ach = k["algorithmic_bytes_per_launch"] / t / 1e9
    return dict(bound="hbm", achieved=ach, peak=PEAK_HBM_GBS, unit="GB/s", frac=ach / PEAK_HBM_GBS, traffic=traffic,
                kernel=name, avg_launch_us=k["avg_launch_us"],
                algorithmic_bytes_per_launch=k["algorithmic_bytes_per_launch"])


# ---------------------------------------------------- HBM byte counters ----
CSRC = os.path.join(ROOT, "paper_1807_01702_amd", "csrc")
SHARED_SOURCES = ["common.hpp", "kernels.hpp", "mfma.hpp", "tiles.hpp"]
CLASS_SOURCES = {"conv1x1": ["conv1x1.hip", "conv_rows.hip"], "conv3x3": ["conv3x3.hip", "conv_rows.hip"],
                 "wgrad1x1": ["conv_wgrad.hip"], "wgrad3x3": ["conv_wgrad.hip"],
                 "stats_sweep": ["bn_kernels.hip"], "elementwise": ["bn_kernels.hip"],
                 "stats_combine": ["bn_kernels.hip"], "splitk_sum": ["bn_kernels.hip"], "pool": ["bn_kernels.hip"],
                 "copy": ["bn_kernels.hip"], "weight_pack": ["conv_rows.hip"], "stem_conv": ["net_ends.hip"],
                 "stem_wgrad": ["net_ends.hip"], "maxpool": ["net_ends.hip"], "head": ["net_ends.hip"]}


def kernel_class(name):
    """Kernel class (as in the launch trace) of a profiler kernel name."""
    n = name.replace("void ", "")
    m = re.search(r"bnr::(k_\w+)(<([^>]*)>)?", n)
    if not m:
        return None
    k, targs = m.group(1), [t.strip() for t in (m.group(3) or "").split(",")]
    if k == "k_conv1x1":
        return "conv1x1"
    if k == "k_conv3x3":
        return "conv3x3"
    if k == "k_conv_rows":
        return "conv1x1" if len(targs) > 1 and targs[1] == "1" else "conv3x3"
    if k in ("k_wgrad_tr", "k_wgrad"):
        taps = targs[0] if k == "k_wgrad_tr" else (targs[1] if len(targs) > 1 else "")
        return "wgrad1x1" if taps == "1" else "wgrad3x3"
    return {"k_stats_partial": "stats_sweep", "k_elementwise": "elementwise", "k_addrelu_bwd": "elementwise",
            "k_stats_combine_one": "stats_combine", "k_stats_combine1": "stats_combine",
            "k_stats_combine2": "stats_combine", "k_sum_partials1": "splitk_sum", "k_sum_partials2": "splitk_sum",
            "k_bwd_tail": "splitk_sum", "k_loss_mean": "head",
            "k_avgpool2": "pool", "k_avgpool2_bwd": "pool", "k_copy16": "copy",
            "k_pack_weights": "weight_pack", "k_stem_conv": "stem_conv", "k_stem_conv_f32": "stem_conv",
            "k_stem_wgrad": "stem_wgrad", "k_stem_wgrad_f32": "stem_wgrad", "k_maxpool_fwd": "maxpool",
            "k_maxpool_bwd": "maxpool", "k_head_pool": "head", "k_fc_gemm": "head", "k_softmax_ce": "head",
            "k_colsum": "head", "k_head_bn_bwd": "head"}.get(k)


def sources_sha(cls):
    h = hashlib.sha256()
    for f in CLASS_SOURCES.get(cls, []) + SHARED_SOURCES:
        with open(os.path.join(CSRC, f), "rb") as fh:
            h.update(f.encode() + b"\0" + fh.read())
    return h.hexdigest()


def _counter_rows(d, counter):
    out = []
    for path in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
        with open(path) as fh:
            for r in csv.DictReader(fh):
                if r["Counter_Name"] == counter:
                    out.append((r["Kernel_Name"], float(r["Counter_Value"]) * 1024.0))   # KiB -> bytes
    return out


def summarize_pmc(fetch_dir, write_dir, workload, copy_mb, bench_json=None):
    """Per kernel class: counter bytes per launch, scaled by the calibration
    copy, and (bench_json: a bench line of the same tree) the algorithmic
    bytes per launch the library's launchers account and the ratio."""
    fetch, write = _counter_rows(fetch_dir, "FETCH_SIZE"), _counter_rows(write_dir, "WRITE_SIZE")
    expected = copy_mb * 1024.0 * 1024.0
    fc = [v for n, v in fetch if kernel_class(n) == "copy"]
    wc = [v for n, v in write if kernel_class(n) == "copy"]
    if not fc or not wc:
        raise SystemExit("no calibration copy in the counter runs (use --calib-copy-mb)")
    f_scale, w_scale = expected / fc[-1], expected / wc[-1]
    agg = {}
    for rows, key in ((fetch, "fetch"), (write, "write")):
        for n, v in rows:
            c = kernel_class(n)
            if c is None or c == "copy":
                continue
            a = agg.setdefault(c, {"fetch": [], "write": []})
            a[key].append(v)
    classes = {}
    for c, a in sorted(agg.items()):
        if not a["fetch"] or not a["write"]:
            continue
        fb = sum(a["fetch"]) / len(a["fetch"]) * f_scale
        wb = sum(a["write"]) / len(a["write"]) * w_scale
        classes[c] = {"launches": len(a["fetch"]), "fetch_bytes_per_launch": fb, "write_bytes_per_launch": wb,
                      "bytes_per_launch": fb + wb, "sources_sha256": sources_sha(c)}
    if bench_json:
        with open(bench_json) as fh:
            kern = json.loads(fh.read().strip().splitlines()[-1])["kernels"]
        for c, v in classes.items():
            if c in kern:
                v["algorithmic_bytes_per_launch"] = kern[c]["algorithmic_bytes_per_launch"]
                v["counter_over_algorithmic"] = v["bytes_per_launch"] / kern[c]["algorithmic_bytes_per_launch"]
    return {"workload": workload, "calibration": {"copy_bytes": expected, "fetch_counted": fc[-1],
                                                  "write_counted": wc[-1], "fetch_scale": f_scale,
                                                  "write_scale": w_scale},
            "classes": classes}


def summarize_step_bytes(fetch_dir, write_dir, copy_mb, steps):
    """HBM bytes per step of a profile-only run: FETCH_SIZE + WRITE_SIZE of
    every library kernel dispatch (the calibration copy excluded), each
    counter scaled by expected / counted bytes of the calibration copy,
    divided by the number of steps the run made (warm-up included)."""
    out = {}
    for d, counter in ((fetch_dir, "FETCH_SIZE"), (write_dir, "WRITE_SIZE")):
        rows = []
        for path in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
            with open(path) as fh:
                rows += [r for r in csv.DictReader(fh) if r["Counter_Name"] == counter]
        rows.sort(key=lambda r: int(r["Dispatch_Id"]))
        lib = [(kernel_class(r["Kernel_Name"]), float(r["Counter_Value"]) * 1024.0) for r in rows
               if kernel_class(r["Kernel_Name"]) is not None]
        if not lib or lib[-1][0] != "copy":
            raise SystemExit("the last library dispatch must be the calibration copy (--calib-copy-mb)")
        scale = copy_mb * 1024.0 * 1024.0 / lib[-1][1]
        out[counter] = {"bytes_per_step": sum(v for _, v in lib[:-1]) * scale / steps, "scale": scale}
    out["total_bytes_per_step"] = out["FETCH_SIZE"]["bytes_per_step"] + out["WRITE_SIZE"]["bytes_per_step"]
    return out


ABLATION_ROWS = [("unfused", "unfused chain (BASELINE: two-pass statistics, BN, ReLU, CONV sweeps)"),
                 ("unfused_rcf", "ReLU-CONV fusion (RCF)"),
                 ("unfused_rcf_mvf", "RCF + mean/variance fusion (MVF)"),
                 ("fused_o2", "BN fission-n-fusion with the stored O2' sweep (the paper's BNFF)"),
                 ("fused_no_icf", "BN fission-n-fusion, z recomputed from x (BNFF)"),
                 ("fused", "BNFF + inter-composite-layer fusion (ICF)")]


def summarize_ablation(run_dir, workload, copy_mb, steps, bench_json=None):
    """HBM bytes per step of every variant with counter runs under run_dir,
    beside the bytes model and (bench_json) the variant's time: writes
    profiles/hbm_bytes_per_step_<workload>.json (with the SHA-256 of all
    kernel sources) and returns a markdown table."""
    from paper_1807_01702_amd import bytes_model, synth
    cls, recipe, kw = WORKLOADS[workload]
    model = bytes_model.for_workload(workload, getattr(synth, recipe)(seed=0, **kw))
    abl = {}
    if bench_json:
        with open(bench_json) as fh:
            abl = json.loads(fh.read().strip().splitlines()[-1])["ablation"]
    h = hashlib.sha256()
    for f in sorted(os.listdir(CSRC)):
        with open(os.path.join(CSRC, f), "rb") as fh:
            h.update(f.encode() + b"\0" + fh.read())
    out = {"workload": workload, "sources_sha256": h.hexdigest(), "variants": {}}
    for v, _ in ABLATION_ROWS:
        fd, wd = os.path.join(run_dir, "sb_f_" + v), os.path.join(run_dir, "sb_w_" + v)
        if not (os.path.isdir(fd) and os.path.isdir(wd)):
            continue
        sb = summarize_step_bytes(fd, wd, copy_mb, steps)
        out["variants"][v] = {"counter_bytes_per_step": sb["total_bytes_per_step"],
                              "fetch_bytes_per_step": sb["FETCH_SIZE"]["bytes_per_step"],
                              "write_bytes_per_step": sb["WRITE_SIZE"]["bytes_per_step"],
                              "model_bytes_per_step": model.get(v),
                              "ms_per_step": abl.get(v, {}).get("ms_per_step")}
    with open(os.path.join(ROOT, "profiles", "hbm_bytes_per_step_%s.json" % workload), "w") as fh:
        json.dump(out, fh, indent=1, sort_keys=True)
    base = out["variants"].get("unfused", {})
    rows = ["| variant | HBM GB/step (counters) | model GB/step | counters / model | vs unfused | ms/step | "
            "speedup vs unfused |", "|---|---|---|---|---|---|---|"]
    for v, label in ABLATION_ROWS:
        r = out["variants"].get(v)
        if not r:
            continue
        mb, ms = r["model_bytes_per_step"], r["ms_per_step"]
        rows.append("| %s | %.2f | %s | %s | %.2f | %s | %s |" % (
            label, r["counter_bytes_per_step"] / 1e9, "%.2f" % (mb / 1e9) if mb else "-",
            "%.2f" % (r["counter_bytes_per_step"] / mb) if mb else "-",
            r["counter_bytes_per_step"] / base["counter_bytes_per_step"] if base else float("nan"),
            "%.3f" % ms if ms else "-",
            "%.2fx" % (base["ms_per_step"] / ms) if (ms and base.get("ms_per_step")) else "-"))
    return "\n".join(rows)


def summarize_bench(bench_json):
    """Markdown: headline figures of a bench line, and per kernel class the
    HIP-event timings of the traced eager steps, warm and with every library
    call preceded by a copy that evicts L2 and the Infinity Cache."""
    with open(bench_json) as fh:
        b = json.loads(fh.read().strip().splitlines()[-1])
    r = b["roofline"]
    out = ["Workload: %s, batch %d." % (b["config"]["workload"], b["config"]["global_batch"]),
           "Bench line: %s = %.0f %s (%.3f ms/step, %s); unfused %.3f ms/step (%.2fx)." % (
        b["metric"], b["value"], b["unit"], b["ms_per_step"], "graph replay" if b["config"].get("graph") else "eager",
        b["unfused"]["ms_per_step"], b["speedup_vs_unfused"]),
        "Dominant kernel class `%s`: %.1f us per launch, %.1f MB algorithmic -> %.0f GB/s = %.3f of %.0f GB/s%s." % (
        r["kernel"], r["avg_launch_us"], r.get("algorithmic_bytes_per_launch", 0) / 1e6, r["achieved"], r["frac"],
        r["peak"], "; counters %.1f MB per launch" % (r["traffic"] / 1e6) if r.get("traffic") else "")]
    cpu = b.get("cpu_baseline")
    if cpu:
        out.append("CPU baseline (the fp64 oracle): %.2f %s on %d threads (%s)." % (cpu["value"], cpu["unit"],
                                                                                  cpu["cores"], cpu["sample"]))
    cold = (b.get("cold_cache") or {}).get("kernels", {})
    out += ["", "| class | launches/step | ms/step | avg us | algorithmic MB | GB/s | of 8 TB/s | cold avg us | "
            "cold / warm |", "|---|---|---|---|---|---|---|---|---|"]
    for k, v in sorted(b["kernels"].items(), key=lambda kv: -kv[1]["ms_per_step"]):
        c = cold.get(k)
        out.append("| %s | %.1f | %.3f | %.1f | %.1f | %.0f | %.2f | %s | %s |" % (
            k, v["launches_per_step"], v["ms_per_step"], v["avg_launch_us"], v["algorithmic_bytes_per_launch"] / 1e6,
            v["achieved_GBps"] or 0, (v["achieved_GBps"] or 0) / PEAK_HBM_GBS,
            "%.1f" % c["avg_launch_us"] if c else "-", "%.3f" % (c["avg_launch_us"] / v["avg_launch_us"]) if c else "-"))
    if cold:
        out.append("")
        out.append("Cold: %d MiB copied (read and written) before every library call of the step, so no operand is "
                   "in L2 or the 256 MB Infinity Cache when a kernel starts." % b["cold_cache"]["flush_mb"])
    return "\n".join(out)


def summarize_mfma(pmc_dir, dtype="bf16"):
    """Markdown table per kernel class from a rocprofv3 --pmc run with
    SQ_VALU_MFMA_BUSY_CYCLES, SQ_INSTS_VALU_MFMA_MOPS_BF16 (or _F32) and
    GRBM_GUI_ACTIVE: matrix-core FLOPs (MOPS x 512), their rate over the
    dispatches' own durations (timestamps) against the dense peak, and the
    matrix-core busy fraction busy / (GUI-active cycles per XCD x SIMDs).
    GRBM_GUI_ACTIVE is reported summed over the 8 XCDs."""
    mops = "SQ_INSTS_VALU_MFMA_MOPS_BF16" if dtype == "bf16" else "SQ_INSTS_VALU_MFMA_MOPS_F32"
    disp = {}
    for path in glob.glob(os.path.join(pmc_dir, "**", "*counter_collection.csv"), recursive=True):
        with open(path) as fh:
            for r in csv.DictReader(fh):
                d = disp.setdefault((path, r["Dispatch_Id"]), {"name": r["Kernel_Name"],
                                                               "dur": (int(r["End_Timestamp"]) -
                                                                       int(r["Start_Timestamp"])) * 1e-9})
                d[r["Counter_Name"]] = float(r["Counter_Value"])
    agg = {}
    for d in disp.values():
        c = kernel_class(d["name"])
        if c is None or "GRBM_GUI_ACTIVE" not in d:
            continue
        a = agg.setdefault(c, [0, 0.0, 0.0, 0.0, 0.0])
        a[0] += 1
        a[1] += d.get(mops, 0.0) * 512
        a[2] += d["dur"]
        a[3] += d.get("SQ_VALU_MFMA_BUSY_CYCLES", 0.0)
        a[4] += d["GRBM_GUI_ACTIVE"] / 8 * 1024
    peak = PEAK_MFMA_TFS[dtype]
    out = ["| class | dispatches | matrix-core TFLOP | time ms | TFLOP/s | of %.0f TFLOP/s peak | busy fraction |"
           % peak, "|---|---|---|---|---|---|---|"]
    for c, (n, fl, t, busy, cyc) in sorted(agg.items(), key=lambda kv: -kv[1][2]):
        if fl <= 0:
            continue
        out.append("| %s | %d | %.3f | %.3f | %.1f | %.3f | %.3f |" % (c, n, fl / 1e12, t * 1e3, fl / t / 1e12,
                                                                    fl / t / 1e12 / peak, busy / cyc))
    return "\n".join(out)


def summarize_lds(pmc_dir):
    """Markdown table per kernel class from a rocprofv3 --pmc run with
    SQ_INSTS_LDS and SQ_LDS_BANK_CONFLICT: LDS instructions and bank-conflict
    cycles per dispatch (summed over the dispatch's waves), and conflict
    cycles per LDS instruction."""
    disp = {}
    for path in glob.glob(os.path.join(pmc_dir, "**", "*counter_collection.csv"), recursive=True):
        with open(path) as fh:
            for r in csv.DictReader(fh):
                d = disp.setdefault((path, r["Dispatch_Id"]), {"name": r["Kernel_Name"]})
                d[r["Counter_Name"]] = float(r["Counter_Value"])
    agg = {}
    for d in disp.values():
        c = kernel_class(d["name"])
        if c is None or "SQ_INSTS_LDS" not in d:
            continue
        a = agg.setdefault(c, [0, 0.0, 0.0])
        a[0] += 1
        a[1] += d["SQ_INSTS_LDS"]
        a[2] += d.get("SQ_LDS_BANK_CONFLICT", 0.0)
    out = ["| class | dispatches | LDS instructions per dispatch | bank-conflict cycles per dispatch | "
           "conflict cycles per LDS instruction |", "|---|---|---|---|---|"]
    for c, (n, li, bc) in sorted(agg.items(), key=lambda kv: -kv[1][1]):
        if li <= 0:
            continue
        out.append("| %s | %d | %.0f | %.0f | %.2f |" % (c, n, li / n, bc / n, bc / li))
    return "\n".join(out)


def traffic_for(workload, cls):
    """Counter bytes per launch of a kernel class, if measured on the current sources."""
    path = os.path.join(ROOT, "profiles", "hbm_traffic_%s.json" % workload)
    try:
        with open(path) as fh:
            d = json.load(fh)
        c = d["classes"][cls]
    except (OSError, KeyError, ValueError):
        return None
    return c["bytes_per_launch"] if c.get("sources_sha256") == sources_sha(cls) else None


def _short(n):
    n = re.sub(r"\(.*", "", n)
    return n.replace("void ", "").replace("unsigned short", "bf16")


def summarize_trace(stats_csv, steps, workload, bench_json=None):
    """Markdown tables: rocprofv3 --stats per kernel, per class, and the byte
    counters of profiles/hbm_traffic_<workload>.json against the algorithmic
    bytes of a bench line (if given)."""
    with open(stats_csv) as fh:
        rows = list(csv.DictReader(fh))
    tot = sum(float(r["TotalDurationNs"]) for r in rows)
    out = ["Steps in the trace: %d (warm-up included). Kernel time per step: %.3f ms." % (steps, tot / steps / 1e6),
           "", "| kernel | launches/step | avg us | min us | max us | share |", "|---|---|---|---|---|---|"]
    for r in sorted(rows, key=lambda r: -float(r["TotalDurationNs"])):
        out.append("| `%s` | %.1f | %.1f | %.1f | %.1f | %.1f%% |" % (
            _short(r["Name"]), int(r["Calls"]) / steps, float(r["AverageNs"]) / 1e3, float(r["MinNs"]) / 1e3,
            float(r["MaxNs"]) / 1e3, 100 * float(r["TotalDurationNs"]) / tot))
    groups = {}
    for r in rows:
        a = groups.setdefault(kernel_class(r["Name"]) or _short(r["Name"])[:40], [0, 0.0])
        a[0] += int(r["Calls"])
        a[1] += float(r["TotalDurationNs"])
    out += ["", "By kernel class (the classes of the bench line's `kernels`):", "",
            "| class | launches/step | avg us | ms/step |", "|---|---|---|---|"]
    for g, (n, t) in sorted(groups.items(), key=lambda kv: -kv[1][1]):
        out.append("| %s | %.1f | %.1f | %.3f |" % (g, n / steps, t / n / 1e3, t / steps / 1e6))
    path = os.path.join(ROOT, "profiles", "hbm_traffic_%s.json" % workload)
    if os.path.exists(path):
        with open(path) as fh:
            tr = json.load(fh)
        alg = {}
        if bench_json:
            with open(bench_json) as fh:
                alg = {k: v["algorithmic_bytes_per_launch"] for k, v in json.loads(fh.read())["kernels"].items()}
        cal = tr["calibration"]
        out += ["", "HBM bytes per launch from the FETCH_SIZE and WRITE_SIZE counter runs, each scaled by "
                "expected / counted bytes of a %d MiB `bnr_hbm_copy` in the same run (fetch x%.3f, write x%.3f):"
                % (cal["copy_bytes"] / 2 ** 20, cal["fetch_scale"], cal["write_scale"]), "",
                "| class | fetch MB | write MB | total MB | algorithmic MB | total / algorithmic |",
                "|---|---|---|---|---|---|"]
        for c, v in sorted(tr["classes"].items(), key=lambda kv: -kv[1]["bytes_per_launch"]):
            a = alg.get(c)
            out.append("| %s | %.1f | %.1f | %.1f | %s | %s |" % (
                c, v["fetch_bytes_per_launch"] / 1e6, v["write_bytes_per_launch"] / 1e6, v["bytes_per_launch"] / 1e6,
                "%.1f" % (a / 1e6) if a else "-", "%.2f" % (v["bytes_per_launch"] / a) if a else "-"))
    return "\n".join(out)


def bn_passes(torch, mb, reps):
    """Markdown table: the standalone BN sweeps (the passes BN fission/fusion
    keeps where a BN's producer or reader is not a CONV) on bf16 tensors of
    about `mb` MB ([m][256]), each launch timed by the library's HIP events,
    achieved rate = the launcher's algorithmic bytes / event time, against
    8 TB/s; the calibration copy beside them."""
    from paper_1807_01702_amd import bnr as B
    c = 256
    m = mb * 1000 * 1000 // (2 * c)
    bf = dict(dtype=torch.bfloat16, device="cuda")
    f32 = dict(dtype=torch.float32, device="cuda")
    gen = torch.Generator(device="cuda").manual_seed(0)
    x, y, g = (torch.randn((m, c), generator=gen, **f32).to(torch.bfloat16) for _ in range(3))
    out, gm, dx = (torch.empty((m, c), **bf) for _ in range(3))
    bn = B.BN(torch.ones(c, **f32), torch.zeros(c, **f32), 1e-5)
    dg, db, al, bp = (torch.randn(c, generator=gen, **f32) * 0.01 for _ in range(4))
    cs, cd = torch.empty((m, c), **bf), torch.empty((m, c), **bf)
    passes = [("statistics sweep (sum x, sum x^2)", lambda: B.bnr_bn_stats(x, bn)),
              ("BN input gradient (dy, x -> dx)", lambda: B.bnr_bn_dx(g, x, bn, dg, db, dx)),
              ("summed-gradient input gradient (G, x -> dX)", lambda: B.bnr_split_dx(g, x, bn, al, bp, dx)),
              ("BN + add + ReLU (y, id -> out)", lambda: B.bnr_bn_add_relu_fwd(y, bn, x, out)),
              ("its backward (g, out, y -> gm, sums)", lambda: B.bnr_bn_add_relu_bwd(g, out, y, bn, gm, dg, db)),
              ("calibration copy", lambda: B.bnr_hbm_copy(cs, cd))]
    rows = ["| pass | kernel | launches | avg us | algorithmic MB | TB/s | of 8 TB/s |", "|---|---|---|---|---|---|---|"]
    for label, f in passes:
        for _ in range(3):
            f()
        torch.cuda.synchronize()
        B.bnr_trace_begin(0xF, 100000)
        for _ in range(reps):
            f()
        torch.cuda.synchronize()
        agg = {}
        for name, ms, by, fl in B.bnr_trace_end(100000):
            a = agg.setdefault(name, [0, 0.0, 0.0])
            a[0] += 1
            a[1] += ms
            a[2] += by
        for name, (n, ms, by) in sorted(agg.items(), key=lambda kv: -kv[1][1]):
            rate = by / (ms * 1e-3) / 1e12
            rows.append("| %s | %s | %d | %.1f | %.1f | %.2f | %.2f |" % (label, name, n, 1e3 * ms / n, by / n / 1e6,
                                                                       rate, rate * 1e3 / PEAK_HBM_GBS))
    return ("Tensors [%d][%d] bf16 (%.1f MB each); %d timed calls per pass after 3 warm-up calls.\n\n" %
            (m, c, m * c * 2 / 1e6, reps)) + "\n".join(rows)


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
    elif args.workload == "densenet121":
        n = 1                     # bounded sample: one image of the whole network (per-image cost is batch independent)
        d = synth.densenet(seed=0, n=n)
        t0 = time.perf_counter()
        _, c = OC.densenet_fwd(d, d["eps"], rnd)
        OC.densenet_bwd(c, rnd)
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
    if args.summarize_pmc:
        if args.calib_copy_mb <= 0:
            raise SystemExit("--summarize-pmc needs the --calib-copy-mb value the counter runs used")
        out = summarize_pmc(args.summarize_pmc[0], args.summarize_pmc[1], args.workload, args.calib_copy_mb,
                            args.bench_json)
        path = os.path.join(ROOT, "profiles", "hbm_traffic_%s.json" % args.workload)
        with open(path, "w") as fh:
            json.dump(out, fh, indent=1, sort_keys=True)
        print(json.dumps(out["classes"]))
        return
    if args.summarize_mfma:
        print(summarize_mfma(args.summarize_mfma))
        return
    if args.summarize_lds:
        print(summarize_lds(args.summarize_lds))
        return
    if args.summarize_step_bytes:
        if args.calib_copy_mb <= 0:
            raise SystemExit("--summarize-step-bytes needs the --calib-copy-mb value the counter runs used")
        print(json.dumps(summarize_step_bytes(args.summarize_step_bytes[0], args.summarize_step_bytes[1],
                                              args.calib_copy_mb, args.steps + args.warmup)))
        return
    if args.summarize_ablation:
        if args.calib_copy_mb <= 0:
            raise SystemExit("--summarize-ablation needs the --calib-copy-mb value the counter runs used")
        print(summarize_ablation(args.summarize_ablation, args.workload, args.calib_copy_mb, args.steps + args.warmup,
                                 args.bench_json))
        return
    if args.summarize_bench:
        print(summarize_bench(args.summarize_bench))
        return
    if args.summarize_trace:
        print(summarize_trace(args.summarize_trace[0], int(args.summarize_trace[1]), args.workload, args.bench_json))
        return
    if args.gpus != 1:
        print("bench.py measures one GPU: the library has no multi-GPU path (run with --gpus 1)", file=sys.stderr)
        sys.exit(2)
    import torch
    if args.bn_passes:
        print(bn_passes(torch, args.bn_passes, args.steps))
        return
    from paper_1807_01702_amd import bytes_model
    torch.cuda.set_device(0)
    data, wls = build_workloads(args, torch)
    res = {}
    for name, wl in wls.items():
        ms, wall, _ = timed_steps(torch, wl, args.steps, args.warmup, not args.no_graph)
        res[name] = dict(ms=ms, wall=wall, images=wl.images)
    if args.profile_only:
        if args.calib_copy_mb > 0:
            from paper_1807_01702_amd import bnr as B
            nb = args.calib_copy_mb * 1024 * 1024
            src = torch.ones(nb // 4, dtype=torch.float32, device="cuda")
            dst = torch.empty_like(src)
            torch.cuda.synchronize()
            B.bnr_hbm_copy(src, dst)
            torch.cuda.synchronize()
        print(json.dumps({k: v["ms"] for k, v in res.items()}))
        return
    dtype = "bf16" if data.get("bf16") else "f32"
    kernels = traced_kernels(torch, wls["fused"], args.steps) if "fused" in wls else None
    cold = (traced_kernels(torch, wls["fused"], min(args.steps, 5), args.flush_mb)
            if "fused" in wls and args.flush_mb > 0 else None)
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
                                                "identity shortcuts",
                                "densenet121": "DenseNet-121 (7x7/2 CONV + 3x3/2 max pooling, dense blocks of "
                                               "6/12/24/16 layers, growth 32, compression-1/2 transitions, "
                                               "1000-way FC + softmax cross-entropy)"}[args.workload],
                   "global_batch": fused["images"] if fused else unf["images"],
                   "image_hw": 224 if args.workload == "densenet121" else 56,
                   "graph": not args.no_graph},
        "unfused": {"images_per_s": unf["images"] / (unf["ms"] / 1e3), "ms_per_step": unf["ms"]} if unf else None,
        "fused_no_icf": ({"images_per_s": noicf["images"] / (noicf["ms"] / 1e3), "ms_per_step": noicf["ms"],
                          "algorithmic_bytes": model.get("fused_no_icf")} if noicf else None),
        "speedup_vs_unfused": (unf["ms"] / fused["ms"]) if (fused and unf) else None,
        "ablation": {k: {"images_per_s": v["images"] / (v["ms"] / 1e3), "ms_per_step": v["ms"],
                         **({"algorithmic_bytes": model[k]} if k in model else {})}
                     for k, v in res.items()},
        "hbm_bytes_per_step": {"algorithmic_fused": model["fused"], "algorithmic_unfused": model["unfused"]},
        "roofline": roofline(kernels, dtype, args.workload) if kernels else None,
        "kernels": kernels,
        # every library call preceded by a copy that evicts L2 and the Infinity Cache
        "cold_cache": ({"flush_mb": args.flush_mb, "roofline": roofline(cold, dtype, args.workload),
                        "kernels": {k: {"avg_launch_us": v["avg_launch_us"], "ms_per_step": v["ms_per_step"],
                                        "achieved_GBps": v["achieved_GBps"]} for k, v in cold.items()}}
                       if cold else None),
        "cpu_baseline": None if args.no_cpu_baseline else cpu_baseline(args),
    }
    print(json.dumps(line))


if __name__ == "__main__":
    main()
