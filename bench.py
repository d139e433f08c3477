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


def parse():
    p = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawTextHelpFormatter)
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=50)
    p.add_argument("--warmup", type=int, default=10)
    p.add_argument("--net", default="c3d", choices=["c3d", "r2plus1d"])
    p.add_argument("--batch", type=int, default=1)
    p.add_argument("--dtype", default="bf16", choices=["bf16", "f16", "f32"])
    p.add_argument("--rate", type=float, default=3.0, help="whole-stack MAC pruning rate (KGS)")
    p.add_argument("--mode", default="kgs", choices=["kgs", "vanilla"])
    p.add_argument("--group", default="4x4", help="kernel group size g_MxG_N of the masks")
    p.add_argument("--no-graph", action="store_true", help="launch eagerly instead of a HIP graph")
    p.add_argument("--separate-pool", action="store_true",
                   help="run max-pools as their own kernels instead of in the conv epilogue")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--cpu-sample", type=float, default=1.0,
                   help="fraction of every layer's outputs the oracle computes (1 = full clip)")
    p.add_argument("--layer-reps", type=int, default=20)
    p.add_argument("--report", default=None, help="write per-layer results to this JSON file")
    p.add_argument("--profile-layer", default=None,
                   help="only launch this layer's sparse conv --layer-reps times (for rocprofv3)")
    p.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                   help="with --profile-layer: also run a plain device copy of MIB MiB, the "
                        "reference for scaling rocprofv3 FETCH_SIZE / WRITE_SIZE")
    return p.parse_args()


def group_of(args):
    gm, gn = (int(v) for v in args.group.lower().split("x"))
    return gm, gn


def log(*a):
    print(*a, file=sys.stderr, flush=True)


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


def per_layer_ms(torch, stack, reps, stream):
    """Average duration of each layer's conv kernel, launched back to back."""
    out = []
    inputs = {}
    cur = stack.x
    for l, conv in zip(stack.layers, stack.convs):
        inp = stack.bufs[l.input_from] if l.input_from else cur
        res = stack.bufs[l.residual_from] if l.residual_from else None
        fn = (lambda conv=conv, inp=inp, res=res, o=stack.bufs[l.name]: conv(inp, res, out=o))
        fn()
        out.append(time_region(torch, fn, reps, stream))
        cur = stack.pool_bufs.get(l.name, stack.bufs[l.name])
        inputs[l.name] = cur
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


def measured_traffic(layer):
    """HBM bytes per launch of `layer`'s KGS conv from the committed
    rocprofv3 FETCH_SIZE / WRITE_SIZE summaries, or None when no summary
    exists for it or the kernels changed since it was taken."""
    import glob
    for path in glob.glob(os.path.join(ROOT, "profiles", "*.md")):
        with open(path) as fh:
            for line in fh:
                if line.startswith("traffic-json:"):
                    d = json.loads(line.split(":", 1)[1])
                    if d.get("layer") == layer and d.get("source_hash") == library_source_hash():
                        return d["traffic_bytes_per_launch"]
    return None


def profile_layer(args, torch, stream):
    """Launch one layer of the sparse stack back to back (and optionally a
    plain copy of known size) so rocprofv3 sees only these kernels."""
    from paper_2007_09835_amd.stack import Stack
    sparse = Stack(args.net, args.batch, args.dtype, args.mode, args.rate,
                   fuse_pool=not args.separate_pool, group=group_of(args))
    idx = [l.name for l in sparse.layers].index(args.profile_layer)
    l, conv = sparse.layers[idx], sparse.convs[idx]
    inp = torch.randn(conv.desc_for(args.batch).n, l.t, l.h, l.w, l.c_in, device="cuda").abs()
    inp = inp.to(sparse.x.dtype)
    res = torch.zeros_like(sparse.bufs[l.name]) if l.residual_from else None
    fn = lambda: conv(inp, res, out=sparse.bufs[l.name])
    fn()
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
                oracle.conv3d_kgs(x64, w64, mask, 4, 4, b64, None, l.stride, l.pad, l.relu)
            elapsed += time.perf_counter() - t0
        else:
            k = max(1, int(n_out * fraction))
            idx = np.sort(synth.rng_for("cpu-sample", l.name).choice(n_out, size=k, replace=False))
            t0 = time.perf_counter()
            oracle.conv3d_points(x64, w64, idx, None if l.dense else mask, 4, 4, b64, None,
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


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py runs on one GPU only: this build has no multi-GPU path "
              "(clips are independent, so --gpus N would be N copies of this run)",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2007_09835_amd import build, synth
    from paper_2007_09835_amd.stack import Stack

    build.build(force=False)
    torch.cuda.set_device(0)
    stream = torch.cuda.current_stream()

    if args.profile_layer:
        profile_layer(args, torch, stream)
        return

    log("building stacks ...")
    fuse = not args.separate_pool
    sparse = Stack(args.net, args.batch, args.dtype, args.mode, args.rate, fuse_pool=fuse,
                   group=group_of(args))
    dense = Stack(args.net, args.batch, args.dtype, "dense", fuse_pool=fuse)
    l0 = sparse.layers[0]
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
        eager = stack.forward().clone()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            stack.forward()
        g.replay()
        torch.cuda.synchronize()
        replay = stack.bufs[stack.layers[-1].name]
        if not torch.equal(eager, replay):
            raise RuntimeError("graph replay differs from the eager pass")
        return g.replay

    run_sparse = runner(sparse)
    run_dense = runner(dense)
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
            "executed_tflops": 2 * kept / lay_s[i] / 1e9,
            "dense_kernel_tflops": 2 * macs_dense / lay_d[i] / 1e9,
        })
        row = rows[-1]
        log("%-10s %5d->%-5d R=%.2f  kgs %.4f ms (%.0f/%.0f TF eq/exec)  dense %.4f ms (%.0f TF)"
            "  speedup %.2f (%.2f R)" % (l.name, l.c_in, l.c_out, r, lay_s[i],
                                         row["dense_equiv_tflops"], row["executed_tflops"],
                                         lay_d[i], row["dense_kernel_tflops"], row["speedup"],
                                         row["speedup_over_rate"]))

    # Dominant kernel: the sparse-stack layer with the largest duration.
    dom = max(range(len(rows)), key=lambda i: rows[i]["ms_sparse"])
    drow = rows[dom]
    l = sparse.layers[dom]
    kept_flops = 2.0 * (args.batch * l.voxels_out * sparse.convs[dom].info.kept_weights
                        if drow["kgs"] else l.dense_macs(args.batch))
    achieved = kept_flops / (drow["ms_sparse"] * 1e-3) / 1e12
    peak = PEAK_TFLOPS[args.dtype]
    traffic = measured_traffic(l.name) if (args.batch == 1 and args.net == "c3d"
                                           and args.dtype == "bf16" and args.mode == "kgs"
                                           and group_of(args) == (4, 4)) else None
    roofline = {"bound": "mfma", "achieved": round(achieved, 2), "peak": peak, "unit": "TFLOP/s",
                "frac": round(achieved / peak, 4), "traffic": traffic,
                "kernel": "%s conv (%s)" % (l.name, "KGS" if drow["kgs"] else "dense"),
                "flops_per_launch": kept_flops}

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
            "workload": "%s conv stack, %d x 16x112x112 clip, %s %s masks g=%s, whole-stack "
                        "pruning rate %.2fx (conv1 dense)%s"
                        % (args.net.upper(), args.batch, args.dtype, args.mode.upper(),
                           args.group.lower(), rate,
                           ", HIP graph" if not args.no_graph else ", eager launches"),
            "batch": args.batch, "clip": [16, 112, 112], "pruning_rate": round(rate, 4),
        },
        "ms_per_clip": round(ms_sparse / args.batch, 5),
        "executed_tflops": round(dense_flops / rate / (ms_sparse * 1e-3) / 1e12, 3),
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
