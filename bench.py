#!/usr/bin/env python3
"""Benchmark: KGS-sparse C3D conv stack on one MI355X.

A step is one forward pass of the whole hot path over one batch: conv1
(dense kernel), max-pools and the seven KGS layers conv2..conv5b, on a
seeded synthetic 16x112x112 RGB clip (U(0,1)) with Kaiming-normal weights and
per-layer keep counts giving a whole-stack pruning rate of about 3x.  The
same stack with every layer on the dense kernel gives the speedup.  Inputs,
weights and packed blobs are resident in HBM before the timed region; the
whole pass is replayed as one HIP graph.

Prints ONE JSON line (stdout).  Per-layer details go to stderr and, with
--report, to a JSON file.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "KGS conv3d dense-equiv TFLOP/s + ms/clip (C3D 16x112x112); speedup vs dense"
PEAK_TFLOPS = {"bf16": 2500.0, "f16": 2500.0, "f32": 157.3}   # dense MFMA, MI355X spec
HBM_GBPS = 8000.0                                                   # HBM3E, MI355X spec


def parse():
    p = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawTextHelpFormatter)
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=50)
    p.add_argument("--warmup", type=int, default=10)
    p.add_argument("--net", default="c3d", choices=["c3d", "r2plus1d", "s3d"])
    p.add_argument("--batch", type=int, default=1)
    p.add_argument("--dtype", default="bf16", choices=["bf16", "f16", "f32"])
    p.add_argument("--rate", type=float, default=None,
                   help="whole-stack MAC pruning rate (KGS); default 3 (C3D) or 2.1 (S3D)")
    p.add_argument("--mode", default="kgs", choices=["kgs", "vanilla", "dense"],
                   help="masks of the sparse stack (dense: every layer on the dense kernel; "
                        "profiling modes only)")
    p.add_argument("--group", default="4x4", help="kernel group size g_MxG_N of the masks")
    p.add_argument("--no-graph", action="store_true", help="launch eagerly instead of a HIP graph")
    p.add_argument("--clock-warmup", type=float, default=0.5, metavar="SECONDS",
                   help="load the GPU this long before measuring (clock ramp-up)")
    p.add_argument("--streams", type=int, default=2,
                   help="S3D: streams for independent Inception branches (1 = in order; "
                        "2 measured fastest at batch 1)")
    p.add_argument("--separate-pool", action="store_true",
                   help="run max-pools as their own kernels instead of in the conv epilogue")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--cpu-sample", type=float, default=1.0,
                   help="fraction of every layer's outputs the oracle computes (1 = full clip)")
    p.add_argument("--layer-reps", type=int, default=20)
    p.add_argument("--report", default=None, help="write per-layer results to this JSON file")
    p.add_argument("--profile-layer", default=None,
                   help="only launch this layer's sparse conv --layer-reps times (for rocprofv3)")
    p.add_argument("--layer-graph", action="store_true",
                   help="--profile-layer: launch from a HIP graph of --layer-reps launches")
    p.add_argument("--profile-reweight", default=None, metavar="LAYER",
                   help="launch only the reweight pass over this C3D layer's weights "
                        "(bf16, all outputs) --layer-reps times, for rocprofv3")
    p.add_argument("--suite", default=None, metavar="PATH",
                   help="instead of the headline line, run the per-config measurement suite "
                        "(single layers, R(2+1)D, batch-32 rate sweep, warm/cold latency, oracle "
                        "timing) and write a markdown report to PATH (+ PATH.json)")
    p.add_argument("--profile-stack", default=None, metavar="MANIFEST",
                   help="launch every layer of the stack (--net/--batch/--mode) --layer-reps "
                        "times back to back, in order, for rocprofv3; write the dispatch "
                        "manifest (JSON) to MANIFEST")
    p.add_argument("--summarize-profile", default=None, metavar="DIR",
                   help="per-layer markdown table from the rocprofv3 runs of --profile-stack "
                        "under DIR (subdirectories trace, fetch, write, sqa, sqb and "
                        "manifest.json)")
    p.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                   help="with --profile-layer: also run a plain device copy of MIB MiB, the "
                        "reference for scaling rocprofv3 FETCH_SIZE / WRITE_SIZE")
    return p.parse_args()


def group_of(args):
    gm, gn = (int(v) for v in args.group.lower().split("x"))
    return gm, gn


def log(*a):
    print(*a, file=sys.stderr, flush=True)


SPIN_CYCLES = 400000   # ~0.2 ms of GPU spin, longer than the host's enqueue of one launch


def clock_warmup(torch, seconds):
    """Keep the GPU under load for `seconds` before measuring: its clocks ramp
    up over the first fraction of a second of work.  Large bf16 matrix
    products give the load with few kernel launches (short profiler traces)."""
    if seconds <= 0:
        return
    a = torch.ones(8192, 8192, device="cuda", dtype=torch.bfloat16)
    b = torch.ones(8192, 8192, device="cuda", dtype=torch.bfloat16)
    t_end = time.perf_counter() + seconds
    while time.perf_counter() < t_end:
        for _ in range(4):
            torch.mm(a, b)
        torch.cuda.synchronize()
    del a, b


def time_region(torch, fn, steps, stream):
    """Run fn() `steps` times between two events on `stream`; ms per call."""
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(steps):
        fn()
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / steps


def graph_of(torch, fn, reps):
    """A HIP graph holding `reps` back-to-back calls of fn (captured on the
    current stream after one eager call, which allocates any workspace)."""
    fn()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for _ in range(reps):
            fn()
    g.replay()
    torch.cuda.synchronize()
    return g


def layer_roofline(l, conv, batch, ms):
    """Roofline of one conv launch: algorithmic FLOPs (kept MACs x 2) and
    bytes (input read once, kept weights once, bias, output written once,
    residual read once), the bound they give at the MI355X peaks, and the
    fraction of it the measured time `ms` reaches (roofline time / time)."""
    es = 4 if conv.dtype == "f32" else 2
    d = conv.desc_for(batch)
    kept = batch * l.voxels_out * conv.info.kept_weights if conv.sparse else l.dense_macs(batch)
    q = max(d.qt, 1) * max(d.qh, 1) * max(d.qw, 1)
    out_elems = batch * l.voxels_out // q * l.c_out
    nbytes = es * (batch * l.t * l.h * l.w * l.c_in + conv.info.kept_weights + out_elems) + 4 * l.c_out
    if l.residual_from:
        nbytes += es * batch * l.voxels_out * l.c_out
    flops = 2.0 * kept
    t_mma = flops / (PEAK_TFLOPS[conv.dtype] * 1e12)
    t_hbm = nbytes / (HBM_GBPS * 1e9)
    t_roof = max(t_mma, t_hbm)
    return {"flops": flops, "bytes": nbytes, "bound": "mfma" if t_mma >= t_hbm else "hbm",
            "roofline_ms": t_roof * 1e3, "frac": t_roof / (ms * 1e-3)}


def per_layer_ms(torch, stack, reps, stream):
    """Average duration of each layer's conv launch (kernel and split
    reduction), from graph replays of `reps` back-to-back launches: the
    host's per-call cost stays out of the measurement."""
    out = []
    for _, fn in stack.layer_calls():
        g = graph_of(torch, fn, reps)
        out.append(time_region(torch, g.replay, 5, stream) / reps)
        del g
    return out


def library_source_hash():
    """Hash of the HIP library sources (ties a stored traffic measurement to
    the kernels it was taken on)."""
    import hashlib
    h = hashlib.sha256()
    for f in ("rt3d_kernels.hip", "rt3d_host.cpp", "rt3d_internal.h"):
        with open(os.path.join(ROOT, "paper_2007_09835_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def measured_profile(layer, net="c3d", batch=1, mode="kgs", dtype="bf16"):
    """The committed rocprofv3 summary row of `layer` (HBM bytes per launch of
    its conv and split reduction, MFMA work executed over kept), or None when
    no summary exists for it or the kernels changed since it was taken."""
    import glob
    want = {"layer": layer, "net": net, "batch": batch, "mode": mode, "dtype": dtype,
            "source_hash": library_source_hash()}
    for path in sorted(glob.glob(os.path.join(ROOT, "profiles", "*.md"))):
        with open(path) as fh:
            for line in fh:
                if line.startswith("traffic-json:"):
                    d = json.loads(line.split(":", 1)[1])
                    if all(d.get(k) == v for k, v in want.items()):
                        return d
    return None


def measured_traffic(layer, net="c3d", batch=1, mode="kgs", dtype="bf16"):
    """HBM bytes per launch of `layer`'s conv (and split reduction), or None."""
    d = measured_profile(layer, net, batch, mode, dtype)
    return None if d is None else d["traffic_bytes_per_launch"]


def profile_layer(args, torch, stream):
    """Launch one layer of the sparse stack back to back (and optionally a
    plain copy of known size) so rocprofv3 sees only these kernels."""
    from paper_2007_09835_amd import synth
    from paper_2007_09835_amd.stack import make_stack
    sparse = make_stack(args.net, args.batch, args.dtype, args.mode, args.rate,
                        fuse_pool=not args.separate_pool, group=group_of(args))
    idx = [l.name for l in sparse.layers].index(args.profile_layer)
    l, conv = sparse.layers[idx], sparse.convs[idx]
    # The layer's own input in a pass over the benchmark clip (the stack
    # measurement's data: MFMA power, and so the clock, depend on the values).
    l0 = sparse.layers[0]
    sparse.x.copy_(synth.to_dtype(synth.clip_input("bench-clip", args.batch, "uniform01", l0.c_in,
                                                   l0.t, l0.h, l0.w), args.dtype)
                   .permute(0, 2, 3, 4, 1).contiguous().cuda())
    sparse.forward()
    fn = dict((c[0].name, c[1]) for c in sparse.layer_calls())[l.name]
    fn()
    clock_warmup(torch, args.clock_warmup)   # as before the stack measurement
    if args.layer_graph:
        # as the stack measurement launches it: back to back inside a HIP graph
        g = graph_of(torch, fn, args.layer_reps)
        ms = time_region(torch, g.replay, 1, stream) / args.layer_reps
    else:
        ms = time_region(torch, fn, args.layer_reps, stream)
    info = conv.info
    kept = (args.batch * l.voxels_out * info.kept_weights if conv.sparse
            else l.dense_macs(args.batch))
    out = {"layer": l.name, "launches": args.layer_reps, "ms_per_launch": ms,
           "algorithmic_tflops": 2.0 * kept / (ms * 1e-3) / 1e12,
           "workspace_bytes": 0 if conv.workspace(args.batch) is None
           else conv.workspace(args.batch).numel() * 4}
    if args.copy_calibration:
        n = args.copy_calibration * (1 << 20) // 4
        a = torch.ones(n, dtype=torch.float32, device="cuda")
        b = torch.empty_like(a)
        b.copy_(a)
        torch.cuda.synchronize()
        out["copy_bytes_each_way"] = n * 4
    print(json.dumps(out), flush=True)


def _copy_calibration(torch, mib):
    """A plain device copy of `mib` MiB each way (the FETCH_SIZE / WRITE_SIZE
    scale of the profiles)."""
    n = mib * (1 << 20) // 4
    a = torch.ones(n, dtype=torch.float32, device="cuda")
    b = torch.empty_like(a)
    b.copy_(a)
    torch.cuda.synchronize()
    return n * 4


def profile_stack(args, torch, stream):
    """Every conv of the stack launched --layer-reps times back to back (its
    split reduction after each launch when it splits), layer after layer,
    after one pass over the benchmark clip; then a plain copy of known size.
    The manifest lists, per layer, the dispatches of one launch and the
    algorithmic FLOPs and bytes, so a summary can attribute rocprofv3's
    per-dispatch rows to layers by their order."""
    from paper_2007_09835_amd import synth
    from paper_2007_09835_amd.stack import make_stack
    st = make_stack(args.net, args.batch, args.dtype, args.mode, args.rate,
                    fuse_pool=not args.separate_pool, group=group_of(args))
    l0 = st.layers[0]
    st.x.copy_(synth.to_dtype(synth.clip_input("bench-clip", args.batch, "uniform01", l0.c_in,
                                               l0.t, l0.h, l0.w), args.dtype)
               .permute(0, 2, 3, 4, 1).contiguous().cuda())
    layers = []
    for (l, fn), conv in zip(st.layer_calls(), st.convs):
        split = conv.workspace(args.batch) is not None
        roof = layer_roofline(l, conv, args.batch, 1.0)
        i32 = [int(v) for v in __import__("numpy").frombuffer(bytes(conv.info.plan), dtype="int32")[:11]]
        layers.append({"layer": l.name, "kgs": conv.sparse, "dispatches": 2 if split else 1,
                       "variant": int(conv.info.variant), "brick": i32[:3], "slots": i32[8],
                       "mfw": i32[10], "kept_flops": roof["flops"], "bytes": roof["bytes"],
                       "dense_flops": 2.0 * l.dense_macs(args.batch)})
    st.forward()
    torch.cuda.synchronize()
    clock_warmup(torch, args.clock_warmup)
    for (l, fn) in st.layer_calls():
        for _ in range(args.layer_reps):
            fn()
        torch.cuda.synchronize()
    copy_bytes = _copy_calibration(torch, args.copy_calibration or 256)
    man = {"net": args.net, "batch": args.batch, "mode": args.mode, "dtype": args.dtype,
           "rate": st.kept_rate(), "reps": args.layer_reps, "layers": layers,
           "copy_bytes_each_way": copy_bytes, "source_hash": library_source_hash()}
    with open(args.profile_stack, "w") as f:
        json.dump(man, f)
    print(json.dumps({"profile_stack": args.profile_stack, "layers": len(layers)}), flush=True)


def _csv_rows(d, suffix):
    import csv
    import glob
    paths = glob.glob(os.path.join(d, "**", "*" + suffix), recursive=True)
    if not paths:
        raise SystemExit("no %s under %s" % (suffix, d))
    with open(paths[0]) as f:
        return list(csv.DictReader(f))


def _per_dispatch(d, kind):
    """[(kernel name, {counter: value} or duration us)] of every dispatch in
    order (rocprofv3 csv under d)."""
    if kind == "trace":
        rows = _csv_rows(d, "kernel_trace.csv")
        rows.sort(key=lambda r: int(r["Start_Timestamp"]))
        return [(r["Kernel_Name"], (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3)
                for r in rows]
    rows = _csv_rows(d, "counter_collection.csv")
    by = {}
    for r in rows:
        k = int(r["Dispatch_Id"])
        name, vals = by.setdefault(k, (r["Kernel_Name"], {}))
        vals[r["Counter_Name"]] = vals.get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
    return [by[k] for k in sorted(by)]


def summarize_profile(args):
    """Markdown table per layer from the five rocprofv3 runs of --profile-stack."""
    d = args.summarize_profile
    with open(os.path.join(d, "manifest.json")) as f:
        man = json.load(f)
    reps = man["reps"]

    def attribute(kind):
        seq = _per_dispatch(os.path.join(d, kind), kind)
        ours = [x for x in seq if "rt3d" in x[0]]
        other = [x for x in seq if "rt3d" not in x[0]]
        fwd = sum(l["dispatches"] for l in man["layers"])
        pos = fwd
        out = []
        for l in man["layers"]:
            n = l["dispatches"]
            chunk = ours[pos:pos + reps * n]
            pos += reps * n
            out.append(([chunk[i] for i in range(0, len(chunk), n)],
                        [chunk[i] for i in range(1, len(chunk), n)] if n == 2 else []))
        if pos != len(ours):
            raise SystemExit("%s: %d library dispatches, the manifest accounts for %d"
                             % (kind, len(ours), pos))
        return out, other

    def mean(xs, key=None):
        v = [x[1] if key is None else x[1].get(key, 0.0) for x in xs]
        return sum(v) / len(v) if v else 0.0

    trace, _ = attribute("trace")
    fetch, fo = attribute("fetch")
    write, wo = attribute("write")
    sqa, _ = attribute("sqa")
    sqb, _ = attribute("sqb")
    copy = man["copy_bytes_each_way"] / 1024.0
    fscale = copy / max(x[1]["FETCH_SIZE"] for x in fo)
    wscale = copy / max(x[1]["WRITE_SIZE"] for x in wo)
    peak = PEAK_TFLOPS[man["dtype"]]
    lines = ["| layer | map | plan | conv us | reduce us | traffic MB (conv+red) | algorithmic MB | "
             "MfmaUtil % | MFMA exec / kept | VALU / MFMA | LDS / MFMA | LDS conflict | "
             "roofline frac |", "|" + "---|" * 13]
    js = []
    for i, l in enumerate(man["layers"]):
        conv_us = mean(trace[i][0])
        red_us = mean(trace[i][1])
        fb = (mean(fetch[i][0], "FETCH_SIZE") + mean(fetch[i][1], "FETCH_SIZE")) * 1024 * fscale
        wb = (mean(write[i][0], "WRITE_SIZE") + mean(write[i][1], "WRITE_SIZE")) * 1024 * wscale
        a = {k: mean(sqa[i][0], k) for k in sqa[i][0][0][1]}
        a.update({k: mean(sqb[i][0], k) for k in sqb[i][0][0][1]})
        mfma = a.get("SQ_INSTS_MFMA", 0.0)
        gui = a.get("GRBM_GUI_ACTIVE", 1.0)
        util = 100.0 * a.get("SQ_VALU_MFMA_BUSY_CYCLES", 0.0) / max(gui / 8.0 * 1024.0, 1.0)
        # 16x16x32 (16-bit) MFMAs: 16384 FLOP each; 16x16x4 f32: 2048; 4x4x1 f32 (x16 blocks): 512
        per = {"bf16": 16384.0, "f16": 16384.0, "f32": 2048.0}[man["dtype"]]
        exec_ratio = mfma * per / l["kept_flops"] if l["kept_flops"] else 0.0
        t = (conv_us + red_us) * 1e-6
        frac = max(l["kept_flops"] / (peak * 1e12), l["bytes"] / (HBM_GBPS * 1e9)) / t
        plan = "v%d %dx%dx%d/%d mfw%d" % (l["variant"], *l["brick"], l["slots"], l["mfw"])
        lines.append("| %s | %s | %s | %.2f | %.2f | %.2f | %.2f | %.1f | %.2f | %.1f | %.2f | %.2f | %.3f |"
                     % (l["layer"], "KGS" if l["kgs"] else "dense", plan, conv_us, red_us,
                        (fb + wb) / 1e6, l["bytes"] / 1e6, util, exec_ratio,
                        a.get("SQ_INSTS_VALU", 0.0) / max(mfma, 1.0),
                        a.get("SQ_INSTS_LDS", 0.0) / max(mfma, 1.0),
                        a.get("SQ_LDS_BANK_CONFLICT", 0.0) / max(a.get("SQ_LDS_IDX_ACTIVE", 1.0), 1.0),
                        frac))
        js.append({"layer": l["layer"], "kernel": plan, "source_hash": man["source_hash"],
                   "net": man["net"], "batch": man["batch"], "mode": man["mode"],
                   "dtype": man["dtype"], "conv_avg_us": round(conv_us, 3),
                   "reduce_avg_us": round(red_us, 3), "traffic_bytes_per_launch": int(fb + wb),
                   "fetch_scale": round(fscale, 4), "write_scale": round(wscale, 4),
                   "mfma_util_pct": round(util, 2), "mfma_exec_over_kept": round(exec_ratio, 3)})
    print("\n".join(lines))
    print()
    print("Traffic: FETCH_SIZE scaled by %.4f and WRITE_SIZE by %.4f (a plain device copy of %d MiB "
          "each way in the same runs)." % (fscale, wscale, man["copy_bytes_each_way"] >> 20))
    print()
    for j in js:
        print("traffic-json: " + json.dumps(j))


def cpu_baseline(stack, fraction):
    """Time the oracle on a seeded sample of every layer's outputs."""
    import numpy as np

    import oracle
    from paper_2007_09835_amd import synth
    flops = 0.0
    elapsed = 0.0
    total_outputs = 0
    for i, (l, conv, mask) in enumerate(zip(stack.layers, stack.convs, stack.masks)):
        d = synth.layer_params(stack.net, l)
        w64 = synth.to_dtype(d.w, stack.dtype).double().numpy()
        kind = "uniform01" if i == 0 else "halfnormal"
        x64 = synth.to_dtype(synth.clip_input("cpu-" + l.name, stack.batch, kind, l.c_in, l.t, l.h,
                                              l.w), stack.dtype).double().numpy()
        to, ho, wo = l.out_thw
        n_out = stack.batch * l.c_out * to * ho * wo
        b64 = d.bias.astype(np.float32).astype(np.float64)
        if fraction >= 1.0:
            k = n_out
            t0 = time.perf_counter()
            if l.dense:
                oracle.conv3d_dense(x64, w64, b64, None, l.stride, l.pad, l.relu)
            else:
                oracle.conv3d_kgs(x64, w64, mask, *l.g, b64, None, l.stride, l.pad, l.relu)
            elapsed += time.perf_counter() - t0
        else:
            k = max(1, int(n_out * fraction))
            idx = np.sort(synth.rng_for("cpu-sample", l.name).choice(n_out, size=k, replace=False))
            t0 = time.perf_counter()
            oracle.conv3d_points(x64, w64, idx, None if l.dense else mask, *l.g, b64, None,
                                 l.stride, l.pad, l.relu)
            elapsed += time.perf_counter() - t0
        flops += 2.0 * k * l.c_in * l.ks
        total_outputs += k
    return {
        "value": flops / elapsed / 1e12,
        "unit": "TFLOP/s",
        "cores": oracle.num_threads(),
        "kind": "oracle",
        "sample": ("%s (%d outputs, %.1f s); dense-equivalent FLOPs of the sample / oracle "
                   "wall time; pools excluded"
                   % ("every conv layer of one clip in full" if fraction >= 1.0 else
                      "seeded %.0f%% of every conv layer's outputs" % (100 * fraction),
                      total_outputs, elapsed)),
    }


# ---------------------------------------------------------------------------
# Measurement suite (the per-config report; not the headline line)
# ---------------------------------------------------------------------------

def pct(xs, q):
    import numpy as np
    return float(np.percentile(np.asarray(xs), q))


def latency(torch, fn, iters, stream, flush=None):
    """Per-launch latency (ms) over `iters` launches, each bracketed by its
    own events; with `flush`, 1 GiB is written before every launch (outside
    the events) so L2 and the 256 MB MALL start cold.  A spin kernel queued
    ahead of the first event keeps the GPU busy while the host enqueues the
    launch, so the interval holds GPU time only."""
    times = []
    fn()
    torch.cuda.synchronize()
    for _ in range(iters):
        if flush is not None:
            flush()
        torch.cuda._sleep(SPIN_CYCLES)
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        fn()
        e1.record(stream)
        e1.synchronize()
        times.append(e0.elapsed_time(e1))
    return {"p10": pct(times, 10), "p50": pct(times, 50), "p90": pct(times, 90)}


def reweight_layer(torch, layer, dtype, full):
    """Device tensors and a launcher for one reweight pass over `layer`'s
    weights (structured synthetic weights, KGS scope, l2 norm).  `full` adds
    the gradient and proximal outputs to norms / update / mask / penalty."""
    from paper_2007_09835_amd import rt3d, synth
    l = layer
    g = (4, 4)
    desc = rt3d.make_group_desc(l.c_out, l.c_in, l.k, g, dtype, 2, rt3d.RT3D_SCOPE_KGS)
    w64 = synth.unit_scaled_weights(synth.rng_for("bench-reweight", l.name), l.c_out, l.c_in,
                                    l.k, g)
    w_t = synth.to_dtype(w64, dtype)
    w = w_t.cuda()
    units = rt3d.rt3d_group_units(desc)
    P, Q = -(-l.c_out // g[0]), -(-l.c_in // g[1])
    ks = l.k[0] * l.k[1] * l.k[2]
    t = {"pen": torch.ones(units, device="cuda"), "norms": torch.empty(units, device="cuda"),
         "pen_next": torch.empty(units, device="cuda"), "reg": torch.empty(1, device="cuda"),
         "mask": torch.empty((P, Q, ks), dtype=torch.uint8, device="cuda"),
         "ws": torch.zeros(rt3d.rt3d_group_workspace_size(desc) // 4, device="cuda")}
    if full:
        t["grad"] = torch.zeros(w.shape, device="cuda")
        t["w_prox"] = torch.empty_like(w)
    lam, eps, tau, step = 1e-5, 1e-6, 1e-4, 1.0

    def fn():
        rt3d.rt3d_group_reweight(desc, w, t["pen"], lam, eps, tau, step, norms=t["norms"],
                                 pen_next=t["pen_next"], reg=t["reg"], mask=t["mask"],
                                 grad=t.get("grad"), w_prox=t.get("w_prox"), workspace=t["ws"])
    es = w.element_size()
    nw = w.numel()
    nbytes = es * nw + 4 * units + 8 * units + P * Q * ks
    if full:
        nbytes += 8 * nw + es * nw
    return {"fn": fn, "bytes": nbytes, "w_t": w_t, "t": t, "lam": lam, "eps": eps, "tau": tau,
            "step": step, "units": units}


def reweight_suite(torch, stream, iters, flush):
    """Per C3D KGS layer: latency and HBM rate of the reweight pass, checked
    against the oracle (which is also timed, as the CPU baseline)."""
    import numpy as np

    import oracle
    from paper_2007_09835_amd import synth
    rows = []
    md = ["## NEXT #2: reweighted group-lasso penalty (C3D KGS layers, l2, per-position groups)", "",
          "One pass over the layer's weights [M][N][3][3][3] computing norms, penalty factors, "
          "penalty value and mask (`update`), plus the penalty gradient (accumulated fp32) and the "
          "proximal map (`full`). Algorithmic bytes: weights read once, per-unit arrays, mask, and "
          "for `full` the gradient read+write and the proximal output. HBM peak 8000 GB/s. relL2 "
          "of the norms vs the float64 oracle; oracle timed on the host (all threads).", "",
          "| layer | dtype | outputs | weights | warm p50 us | cold p50 us | GB/s (cold) | frac | relL2 | oracle ms |",
          "|---|---|---|---|---|---|---|---|---|---|"]
    for l in synth.c3d_layers():
        if l.dense:
            continue
        for dtype in ("bf16", "f32"):
            for full in (False, True):
                r = reweight_layer(torch, l, dtype, full)
                warm = latency(torch, r["fn"], iters, stream)
                cold = latency(torch, r["fn"], max(iters // 2, 10), stream, flush)
                r["t"]["pen"].fill_(1.0)
                if full:
                    r["t"]["grad"].zero_()
                r["fn"]()
                torch.cuda.synchronize()
                w64 = r["w_t"].double().numpy()
                t0 = time.perf_counter()
                ref = oracle.group_reweight(w64, 4, 4, norm=2, scope=0, lam=r["lam"], eps=r["eps"],
                                            tau=r["tau"], step=r["step"])
                t_or = time.perf_counter() - t0
                got = r["t"]["norms"].double().cpu().numpy()
                err = float(np.linalg.norm(got - ref["norms"].ravel()) /
                            max(np.linalg.norm(ref["norms"]), 1e-30))
                gbs = r["bytes"] / (cold["p50"] * 1e-3) / 1e9
                rows.append({"layer": l.name, "dtype": dtype, "full": full, "bytes": r["bytes"],
                             "warm": warm, "cold": cold, "gbps_cold": gbs,
                             "gbps_warm": r["bytes"] / (warm["p50"] * 1e-3) / 1e9,
                             "relL2_norms": err, "oracle_s": t_or,
                             "oracle_threads": oracle.num_threads()})
                md.append("| %s | %s | %s | %.2f MB | %.1f | %.1f | %.0f | %.3f | %.1e | %.1f |" % (
                    l.name, dtype, "full" if full else "update", r["bytes"] / 1e6, 1e3 * warm["p50"],
                    1e3 * cold["p50"], gbs, gbs / 8000.0, err, 1e3 * t_or))
                log("reweight %s %s %s: warm %.1f us cold %.1f us %.0f GB/s relL2 %.1e" % (
                    l.name, dtype, "full" if full else "update", 1e3 * warm["p50"],
                    1e3 * cold["p50"], gbs, err))
                del r
    md.append("")
    return {"rows": rows, "md": md}


def suite(args, torch, stream):
    import numpy as np

    import oracle
    from paper_2007_09835_amd import layers as L
    from paper_2007_09835_amd import synth
    from paper_2007_09835_amd.stack import make_stack

    scratch = torch.empty(1 << 28, dtype=torch.float32, device="cuda")   # 1 GiB
    flush = lambda: scratch.fill_(1.0)
    clock_warmup(torch, args.clock_warmup)
    iters = max(args.steps, 50)
    out = {"configs": {}}
    md = ["# Measurement suite (MI355X, one GPU)", "",
          "Latencies are per launch from HIP events (p10 / p50 / p90 over %d launches); warm = "
          "back-to-back launches, cold = 1 GiB written before each launch. Dense-equivalent "
          "TFLOP/s = 2 x dense MACs / time; kept = 2 x kept MACs / time." % iters, "",
          "Command: `python bench.py --suite <path>`", ""]
    cores_all = oracle.num_threads()

    def one_layer(tag, l, cfg, dtype, sparse, g=(4, 4)):
        d = synth.layer_params(cfg["tag"], l, w_std=cfg.get("w_std"))
        mask = d.mask if sparse else None
        w_t = synth.to_dtype(d.w, dtype)
        conv = L.Conv3d(l.c_in, l.c_out, (l.t, l.h, l.w), l.k, l.stride, l.pad, w_t,
                        d.bias.astype(np.float32), mask, dtype, g=g)
        x64 = synth.clip_input(cfg["tag"], 1, cfg["x_kind"], l.c_in, l.t, l.h, l.w)
        x_t = synth.to_dtype(x64, dtype)
        x = x_t.permute(0, 2, 3, 4, 1).contiguous().cuda()
        y = torch.empty(conv.out_shape(1), dtype=L.TORCH_DTYPES[dtype], device="cuda")
        fn = lambda: conv(x, out=y)
        warm = latency(torch, fn, iters, stream)
        cold = latency(torch, fn, iters, stream, flush)
        fn()
        torch.cuda.synchronize()
        got = y.permute(0, 4, 1, 2, 3).double().cpu().numpy()
        return conv, d, x_t, got, warm, cold

    def rel(a, b):
        return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-30))

    # Configs 1 and 2: single layers, every variant checked against the oracle.
    rows = []
    for cname, (l, cfg), dtypes, full in (("1", synth.single_layer_small(), ("f32",), True),
                                          ("2", synth.single_layer_conv3b(), ("f32", "bf16"), False)):
        for dtype in dtypes:
            for sparse in (True, False):
                conv, d, x_t, got, warm, cold = one_layer(cname, l, cfg, dtype, sparse)
                w_ref = synth.to_dtype(d.w, dtype).double().numpy()
                x_ref = x_t.double().numpy()
                b_ref = d.bias.astype(np.float32).astype(np.float64)
                mask = d.mask if sparse else None
                if full:
                    t0 = time.perf_counter()
                    ref = (oracle.conv3d_kgs(x_ref, w_ref, mask, 4, 4, b_ref, None, l.stride, l.pad, True)
                           if sparse else oracle.conv3d_dense(x_ref, w_ref, b_ref, None, l.stride, l.pad, True))
                    t_all = time.perf_counter() - t0
                    err = rel(got, ref)
                    n_or = got.size
                else:
                    idx = np.sort(synth.rng_for("suite", cname, dtype).choice(got.size, 4000, replace=False))
                    t0 = time.perf_counter()
                    ref = oracle.conv3d_points(x_ref, w_ref, idx, mask, 4, 4, b_ref, None, l.stride, l.pad, True)
                    t_all = time.perf_counter() - t0
                    err = rel(got.ravel()[idx], ref)
                    n_or = len(idx)
                # one-thread oracle timing on a bounded sample
                idx1 = np.sort(synth.rng_for("suite1", cname, dtype).choice(got.size, min(got.size, 2000), replace=False))
                oracle.set_threads(1)
                t0 = time.perf_counter()
                oracle.conv3d_points(x_ref, w_ref, idx1, mask, 4, 4, b_ref, None, l.stride, l.pad, True)
                t_one = time.perf_counter() - t0
                oracle.set_threads(cores_all)
                dense_macs = l.dense_macs()
                kept = l.voxels_out * conv.info.kept_weights if sparse else dense_macs
                rows.append({"config": cname, "dtype": dtype, "variant": "KGS" if sparse else "dense",
                             "warm": warm, "cold": cold, "relL2": err, "oracle_outputs": n_or,
                             "dense_eq_tflops": 2 * dense_macs / warm["p50"] / 1e9,
                             "kept_tflops": 2 * kept / warm["p50"] / 1e9,
                             "rate": dense_macs / kept,
                             "oracle_s_all_threads_per_output": t_all / n_or,
                             "oracle_s_one_thread_per_output": t_one / len(idx1)})
                log("cfg%s %s %s warm p50 %.4f ms cold p50 %.4f ms relL2 %.2e" %
                    (cname, dtype, rows[-1]["variant"], warm["p50"], cold["p50"], err))
    out["configs"]["1-2"] = rows
    md += ["## Configs 1 and 2: single layers", "",
           "| cfg | dtype | variant | R | warm p10/p50/p90 ms | cold p50 ms | dense-eq TF | kept TF | relL2 vs oracle | oracle us/output (%d thr / 1 thr) |" % cores_all,
           "|---|---|---|---|---|---|---|---|---|---|"]
    for r in rows:
        md.append("| %s | %s | %s | %.2f | %.4f / %.4f / %.4f | %.4f | %.1f | %.1f | %.2e (%d outputs) | %.2f / %.2f |" % (
            r["config"], r["dtype"], r["variant"], r["rate"], r["warm"]["p10"], r["warm"]["p50"],
            r["warm"]["p90"], r["cold"]["p50"], r["dense_eq_tflops"], r["kept_tflops"], r["relL2"],
            r["oracle_outputs"], 1e6 * r["oracle_s_all_threads_per_output"],
            1e6 * r["oracle_s_one_thread_per_output"]))
    md.append("")

    # Configs 3-5: stacks (whole pass in one HIP graph), per-layer warm latency.
    def stack_pair(net, batch, mode, rate, group=(4, 4)):
        sp = make_stack(net, batch, "bf16", mode, rate, group=group)
        dn = make_stack(net, batch, "bf16", "dense", rate, group=group)
        l0 = sp.layers[0]
        x = synth.to_dtype(synth.clip_input("bench-clip", batch, "uniform01", l0.c_in, l0.t, l0.h,
                                            l0.w), "bf16").permute(0, 2, 3, 4, 1).contiguous().cuda()
        sp.x.copy_(x)
        dn.x.copy_(x)
        res = {}
        for name, st in (("kgs", sp), ("dense", dn)):
            for _ in range(2):
                st.forward()
            torch.cuda.synchronize()
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                st.forward()
            res[name] = {"warm": latency(torch, g.replay, iters, stream),
                         "cold": latency(torch, g.replay, max(iters // 5, 10), stream, flush),
                         "layers": per_layer_ms(torch, st, 20, stream)}
            res[name]["roofline"] = [layer_roofline(l, c, batch, ms) for l, c, ms in
                                     zip(st.layers, st.convs, res[name]["layers"])]
        return sp, res

    md += ["## Configs 3-5: stacks (bf16, HIP graph per pass)", "",
           "| workload | R | KGS ms/clip warm p50 (p10-p90) | cold p50 | dense ms/clip warm p50 | speedup | speedup / R | dense-eq TFLOP/s |",
           "|---|---|---|---|---|---|---|---|"]
    sweep = [("C3D batch 1 (cfg 3)", "c3d", 1, "kgs", 3.0, (4, 4)),
             ("C3D batch 1, g=16x4 (NEXT #1)", "c3d", 1, "kgs", 3.0, (16, 4)),
             ("R(2+1)D-18 batch 1 (cfg 4)", "r2plus1d", 1, "kgs", 3.0, (4, 4)),
             ("S3D 16x224x224 batch 1, 2.1x (NEXT #4)", "s3d", 1, "kgs", 2.1, (4, 4))]
    sweep += [("C3D batch 32, KGS %gx (cfg 5)" % r, "c3d", 32, "kgs", r, (4, 4)) for r in (2.0, 3.0, 4.0, 5.0)]
    sweep += [("C3D batch 32, vanilla 3x (cfg 5)", "c3d", 32, "vanilla", 3.0, (4, 4))]
    stacks = []
    for label, net, batch, mode, rate, group in sweep:
        sp, res = stack_pair(net, batch, mode, rate, group)
        R = sp.kept_rate()
        kw, dw = res["kgs"]["warm"]["p50"], res["dense"]["warm"]["p50"]
        entry = {"label": label, "rate": R, "kgs": res["kgs"], "dense": res["dense"],
                 "layers": [l.name for l in sp.layers],
                 "layer_rates": [l.dense_macs(batch) / (batch * l.voxels_out * c.info.kept_weights)
                                 if m is not None else 1.0 for l, c, m in zip(sp.layers, sp.convs, sp.masks)]}
        stacks.append(entry)
        md.append("| %s | %.2f | %.4f (%.4f-%.4f) | %.4f | %.4f | %.2f | %.2f | %.0f |" % (
            label, R, kw / batch, res["kgs"]["warm"]["p10"] / batch, res["kgs"]["warm"]["p90"] / batch,
            res["kgs"]["cold"]["p50"] / batch, dw / batch, dw / kw, dw / kw / R,
            2 * sp.dense_macs() / (kw * 1e-3) / 1e12))
        log("%s: kgs %.4f ms dense %.4f ms (R %.2f)" % (label, kw, dw, R))
        del sp
        torch.cuda.empty_cache()
    md.append("")
    for e in stacks:
        if "batch 32" not in e["label"] and "R(2+1)D" not in e["label"] and "S3D" not in e["label"]:
            continue
        md += ["### %s: per layer (ms per launch, warm)" % e["label"], "",
               "| layer | R | KGS | dense | speedup | speedup / R | KGS exec TF | KGS roofline frac | dense roofline frac |",
               "|---|---|---|---|---|---|---|---|---|"]
        for name, r, ks, ds, kr, dr in zip(e["layers"], e["layer_rates"], e["kgs"]["layers"],
                                           e["dense"]["layers"], e["kgs"]["roofline"],
                                           e["dense"]["roofline"]):
            md.append("| %s | %.2f | %.4f | %.4f | %.2f | %.2f | %.0f | %.3f (%s) | %.3f (%s) |" % (
                name, r, ks, ds, ds / ks, ds / ks / r, kr["flops"] / (ks * 1e-3) / 1e12,
                kr["frac"], kr["bound"], dr["frac"], dr["bound"]))
        md.append("")
    out["configs"]["stacks"] = stacks

    # NEXT #2: reweighted group-lasso penalty over every KGS layer of C3D.
    rw = reweight_suite(torch, stream, iters, flush)
    out["reweight"] = rw["rows"]
    md += rw["md"]

    # Context: MIOpen dense conv3d (torch) per C3D layer, batch 1, bf16 channels-last.
    md += ["## Context: torch conv3d (MIOpen), C3D layers, batch 1, bf16 (warm p50 ms)", "",
           "| layer | MIOpen | our dense | our KGS (4x4) |", "|---|---|---|---|"]
    try:
        c3d = next(e for e in stacks if e["label"].startswith("C3D batch 1 (cfg 3)"))
        ctx = []
        for i, l in enumerate(synth.c3d_stack(3.0)):
            x = torch.randn(1, l.c_in, l.t, l.h, l.w, device="cuda", dtype=torch.bfloat16).to(
                memory_format=torch.channels_last_3d)
            w = torch.randn(l.c_out, l.c_in, *l.k, device="cuda", dtype=torch.bfloat16).to(
                memory_format=torch.channels_last_3d)
            b = torch.zeros(l.c_out, device="cuda", dtype=torch.bfloat16)
            fn = lambda: torch.nn.functional.conv3d(x, w, b, l.stride, l.pad)
            for _ in range(3):
                fn()
            t = latency(torch, fn, 20, stream)["p50"]
            ctx.append(t)
            md.append("| %s | %.4f | %.4f | %.4f |" % (l.name, t, c3d["dense"]["layers"][i], c3d["kgs"]["layers"][i]))
        out["miopen_c3d_b1_ms"] = ctx
    except Exception as exc:  # MIOpen unavailable or failing: report, do not abort the suite
        md.append("| (torch conv3d failed: %s) | | | |" % str(exc).splitlines()[0][:80])
    md.append("")
    with open(args.suite, "w") as f:
        f.write("\n".join(md) + "\n")
    with open(args.suite + ".json", "w") as f:
        json.dump(out, f, indent=1)
    log("suite written to %s" % args.suite)


def main():
    args = parse()
    if args.rate is None:
        args.rate = 2.1 if args.net == "s3d" else 3.0
    if args.summarize_profile:
        summarize_profile(args)
        return
    if args.gpus != 1:
        print("bench.py runs on one GPU only: this build has no multi-GPU path "
              "(clips are independent, so --gpus N would be N copies of this run)",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2007_09835_amd import build, synth
    from paper_2007_09835_amd.stack import make_stack

    build.build(force=False)
    torch.cuda.set_device(0)
    stream = torch.cuda.current_stream()

    if args.profile_layer:
        profile_layer(args, torch, stream)
        return
    if args.profile_stack:
        profile_stack(args, torch, stream)
        return
    if args.mode == "dense":
        sys.exit("--mode dense selects the profiled stack; the benchmark always times both")
    if args.profile_reweight:
        layer = next(l for l in synth.c3d_layers() if l.name == args.profile_reweight)
        r = reweight_layer(torch, layer, "bf16", True)
        clock_warmup(torch, args.clock_warmup)
        ms = time_region(torch, r["fn"], args.layer_reps, stream)
        out = {"reweight_layer": layer.name, "launches": args.layer_reps, "ms_per_launch": ms,
               "algorithmic_bytes": r["bytes"], "gbps": r["bytes"] / (ms * 1e-3) / 1e9}
        if args.copy_calibration:
            n = args.copy_calibration * (1 << 20) // 4
            a = torch.ones(n, dtype=torch.float32, device="cuda")
            torch.empty_like(a).copy_(a)
            torch.cuda.synchronize()
            out["copy_bytes_each_way"] = n * 4
        print(json.dumps(out), flush=True)
        return
    if args.suite:
        suite(args, torch, stream)
        return

    log("building stacks ...")
    fuse = not args.separate_pool
    sparse = make_stack(args.net, args.batch, args.dtype, args.mode, args.rate, fuse_pool=fuse,
                        group=group_of(args), streams=args.streams)
    dense = make_stack(args.net, args.batch, args.dtype, "dense", args.rate, fuse_pool=fuse,
                       streams=args.streams)
    l0 = sparse.layers[0]
    clip_thw = (l0.t, l0.h, l0.w)
    clip = synth.clip_input("bench-clip", args.batch, "uniform01", l0.c_in, l0.t, l0.h, l0.w)
    x = synth.to_dtype(clip, args.dtype).permute(0, 2, 3, 4, 1).contiguous().cuda()
    sparse.x.copy_(x)
    dense.x.copy_(x)
    rate = sparse.kept_rate()

    def runner(stack):
        if args.no_graph:
            return lambda: stack.forward()
        for _ in range(3):
            stack.forward()
        torch.cuda.synchronize()
        out = stack.forward()
        eager = out.clone()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            stack.forward()
        out.zero_()
        g.replay()
        torch.cuda.synchronize()
        if not torch.equal(eager, out):
            raise RuntimeError("graph replay differs from the eager pass")
        return g.replay

    run_sparse = runner(sparse)
    run_dense = runner(dense)
    clock_warmup(torch, args.clock_warmup)   # outside the timed region
    for _ in range(args.warmup):
        run_sparse()
        run_dense()
    torch.cuda.synchronize()

    # Timed region: exactly `steps` passes of the sparse stack.
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ms_sparse = time_region(torch, run_sparse, args.steps, stream)
    t1 = time.perf_counter()
    ms_dense = time_region(torch, run_dense, args.steps, stream)
    log("sparse %.4f ms/step (wall %.4f), dense %.4f ms/step"
        % (ms_sparse, (t1 - t0) * 1e3 / args.steps, ms_dense))

    # Per-layer kernel durations (events on the launch stream).
    lay_s = per_layer_ms(torch, sparse, args.layer_reps, stream)
    lay_d = per_layer_ms(torch, dense, args.layer_reps, stream)
    rows = []
    for i, l in enumerate(sparse.layers):
        macs_dense = l.dense_macs(args.batch)
        info = sparse.convs[i].info
        kept = macs_dense if sparse.masks[i] is None else (
            args.batch * l.voxels_out * info.kept_weights)
        r = macs_dense / kept
        rows.append({
            "layer": l.name, "c_in": l.c_in, "c_out": l.c_out, "out_thw": list(l.out_thw),
            "kgs": sparse.masks[i] is not None,
            "ms_sparse": lay_s[i], "ms_dense": lay_d[i], "rate": r,
            "speedup": lay_d[i] / lay_s[i], "speedup_over_rate": lay_d[i] / lay_s[i] / r,
            "dense_equiv_tflops": 2 * macs_dense / lay_s[i] / 1e9,
            "kept_tflops": 2 * kept / lay_s[i] / 1e9,
            "dense_kernel_tflops": 2 * macs_dense / lay_d[i] / 1e9,
            "roofline_sparse": layer_roofline(l, sparse.convs[i], args.batch, lay_s[i]),
            "roofline_dense": layer_roofline(dense.layers[i], dense.convs[i], args.batch, lay_d[i]),
        })
        row = rows[-1]
        log("%-10s %5d->%-5d R=%.2f  kgs %.4f ms (%.0f/%.0f TF eq/kept, %.3f of %s roofline)  "
            "dense %.4f ms (%.0f TF, %.3f)  speedup %.2f (%.2f R)" % (
                l.name, l.c_in, l.c_out, r, lay_s[i], row["dense_equiv_tflops"],
                row["kept_tflops"], row["roofline_sparse"]["frac"],
                row["roofline_sparse"]["bound"], lay_d[i], row["dense_kernel_tflops"],
                row["roofline_dense"]["frac"], row["speedup"], row["speedup_over_rate"]))

    # Dominant kernel: the sparse-stack layer with the largest duration.
    dom = max(range(len(rows)), key=lambda i: rows[i]["ms_sparse"])
    drow = rows[dom]
    l = sparse.layers[dom]
    kept_flops = 2.0 * (args.batch * l.voxels_out * sparse.convs[dom].info.kept_weights
                        if drow["kgs"] else l.dense_macs(args.batch))
    achieved = kept_flops / (drow["ms_sparse"] * 1e-3) / 1e12
    peak = PEAK_TFLOPS[args.dtype]
    prof = (measured_profile(l.name, args.net, args.batch, args.mode, args.dtype)
            if group_of(args) == (4, 4) else None)
    traffic = None if prof is None else prof["traffic_bytes_per_launch"]
    # MFMA work the kernel executes (the union's zero weights included) over
    # the kept MACs, from the same counter summary (SQ_INSTS_MFMA).
    exec_over_kept = None if prof is None else prof.get("mfma_exec_over_kept")
    roofline = {"bound": "mfma", "achieved": round(achieved, 2), "peak": peak, "unit": "TFLOP/s",
                "frac": round(achieved / peak, 4), "traffic": traffic,
                "kernel": "%s conv (%s)" % (l.name, "KGS" if drow["kgs"] else "dense"),
                "flops_per_launch": kept_flops,
                "mfma_exec_over_kept": exec_over_kept,
                "mfma_executed_tflops": (None if exec_over_kept is None
                                         else round(achieved * exec_over_kept, 2))}

    dense_flops = 2.0 * sparse.dense_macs()
    value = dense_flops / (ms_sparse * 1e-3) / 1e12
    result = {
        "metric": METRIC,
        "value": round(value, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_sparse, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": args.dtype,
        "data": "synthetic (seeded clip and Kaiming-normal weights; no dataset or trained model)",
        "config": {
            "workload": "%s conv stack, %d x %s clip, %s %s masks g=%s, whole-stack "
                        "pruning rate %.2fx (%s dense)%s"
                        % (args.net.upper(), args.batch, "x".join(map(str, clip_thw)), args.dtype,
                           args.mode.upper(), args.group.lower(), rate, sparse.layers[0].name,
                           ", HIP graph" if not args.no_graph else ", eager launches"),
            "batch": args.batch, "clip": list(clip_thw), "pruning_rate": round(rate, 4),
        },
        "ms_per_clip": round(ms_sparse / args.batch, 5),
        "kept_tflops": round(dense_flops / rate / (ms_sparse * 1e-3) / 1e12, 3),
        "dense_ms_per_step": round(ms_dense, 5),
        "dense_tflops": round(dense_flops / (ms_dense * 1e-3) / 1e12, 3),
        "speedup_vs_dense": round(ms_dense / ms_sparse, 4),
        "speedup_over_rate": round(ms_dense / ms_sparse / rate, 4),
        "roofline": roofline,
    }
    if not args.no_cpu_baseline:
        log("timing the CPU oracle on a sample ...")
        result["cpu_baseline"] = cpu_baseline(sparse, args.cpu_sample)
    if args.report:
        with open(args.report, "w") as f:
            json.dump({"result": result, "layers": rows}, f, indent=1)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
