#!/usr/bin/env python3
"""Benchmark: one Transolver-3 Physics-Attention layer forward on a 100M-point
volume mesh (C=128, H=8 heads of M=64 slices, dh=16, tau=0.5, bf16 storage,
1M-point tiles and decode chunks) on one MI355X.

A step is the whole layer over the resident mesh: pass 1 over every tile,
the ordered fold + Linear1 + token attention + Linear3, and pass 2 over every
chunk.  x is generated on the device (seeded) before timing; the timed region
covers exactly --steps steps between synchronised HIP events.  The line also
carries the dominant kernel's roofline figures (HIP-event launch durations on
the launch stream) and the float64 oracle's throughput on host cores over a
bounded sample.  Prints one JSON line on stdout; progress goes to stderr.

--backward times a float32 training step of the layer instead (forward, then
the backward with the slice weights recomputed per tile) on 2M volume points
(C=128, H=8, M=64, 1M-point tiles), with the backward's roofline against the
float32 matrix peak and the float64 backward oracle as the CPU baseline.

--stack times the 8-block pre-norm Transolver stack (Physics-Attention plus a
4C feed-forward network per block) on a 10M-point car surface (C=256, H=8,
M=64, bf16), with the dominant kernel's roofline and the float64 block oracle
as the CPU baseline.
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "mesh points/s per Physics-Attention layer fwd @100M pts C=128; % roofline"
PEAK_BF16_TFLOPS = 2516.6   # MI355X dense bf16 matrix peak (256 CU x 4096 flop/clk x 2.4 GHz)
PEAK_HBM_GBS = 8000.0


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def kernel_source_hash():
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2602_04940_amd", "csrc")
    for f in sorted(os.listdir(csrc)):
        with open(os.path.join(csrc, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def measured_traffic(kernel: str, launch_points: int):
    """HBM bytes per launch from committed rocprofv3 --pmc summaries, if they were
    taken on the current kernel sources; else None."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        t = json.load(f)
    k = t.get("kernels", {}).get(kernel)
    if not k or t.get("source_hash") != kernel_source_hash() or k.get("points") != launch_points:
        return None
    return k.get("hbm_bytes_per_launch")


CAL_BYTES = 1 << 30  # calibration copy: 1 GiB read, 1 GiB written


def pmc_driver(points: int):
    """Short workload for rocprofv3 --pmc: two layer forwards over `points`
    points (1M-point launches), then one device-to-device copy of CAL_BYTES whose
    counter readings calibrate FETCH_SIZE / WRITE_SIZE."""
    import torch

    from paper_2602_04940_amd import LayerWeights, PhysicsAttention
    from ts3_synth import WORKLOADS, make_weights
    from ts3_synth.device_gen import DeviceVolume
    wl = WORKLOADS["volume_100m_bf16"]
    x = torch.empty((points, wl.C), device="cuda", dtype=torch.bfloat16)
    DeviceVolume(wl.seed, wl.C).fill(x)
    out = torch.empty_like(x)
    lw = LayerWeights(make_weights(wl.C, wl.H, wl.M, wl.dh, seed=0))
    with PhysicsAttention(wl.C, wl.H, wl.M, wl.dh, wl.tau, "bf16", group_span=wl.group_span,
                          max_points=points) as layer:
        for _ in range(2):
            layer.forward(lw, x, tile=wl.tile, chunk=wl.chunk, out=out)
        torch.cuda.synchronize()
    src = torch.empty(CAL_BYTES, device="cuda", dtype=torch.uint8).fill_(1)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    dst.copy_(src)
    torch.cuda.synchronize()
    log("pmc driver done")


def summarize_traffic(fetch_dir: str, write_dir: str, command: str):
    """profiles/traffic.json from two rocprofv3 --pmc runs of --pmc-driver."""
    import csv
    import glob

    def rows(d):
        f = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)
        if not f:
            raise SystemExit(f"no counter_collection.csv under {d}")
        return list(csv.DictReader(open(f[0])))

    out = {"source_hash": kernel_source_hash(), "command": command, "kernels": {}}
    per = {}
    for name, d in (("FETCH_SIZE", fetch_dir), ("WRITE_SIZE", write_dir)):
        rs = [r for r in rows(d) if r["Counter_Name"] == name]
        cal = [r for r in rs if "copyBuffer" in r["Kernel_Name"]][-1]
        factor = CAL_BYTES / (float(cal["Counter_Value"]) * 1024.0)
        out.setdefault("calibration", {})[name] = {"copy_bytes": CAL_BYTES, "counter_kib": float(cal["Counter_Value"]),
                                                  "bytes_per_counted_byte": factor}
        for kname in ("k_slice_accumulate_pc", "k_deslice_w8"):
            vals = [float(r["Counter_Value"]) for r in rs if kname + "<" in r["Kernel_Name"]]
            per.setdefault(kname, {})[name] = (sum(vals) / len(vals), len(vals), factor)
    for kname, d in per.items():
        f_kib, n, f_fac = d["FETCH_SIZE"]
        w_kib, _, w_fac = d["WRITE_SIZE"]
        out["kernels"][kname] = {
            "points": 1_000_000, "dispatches": n, "fetch_kib": f_kib, "write_kib": w_kib,
            "hbm_bytes_per_launch": f_kib * 1024 * f_fac + w_kib * 1024 * w_fac}
    path = os.path.join(ROOT, "profiles", "traffic.json")
    os.makedirs(os.path.dirname(path), exist_ok=True)
    with open(path, "w") as fh:
        json.dump(out, fh, indent=1)
    print(json.dumps(out, indent=1))


def cpu_baseline(x_dev, W, wl, sample):
    """The float64 oracle (as written) on the first `sample` points, host cores."""
    import numpy as np
    from threadpoolctl import threadpool_info

    import oracle
    xs = x_dev[:sample].float().cpu().numpy().astype(np.float64)
    it = 1.0 / wl.tau
    t0 = time.perf_counter()
    st = oracle.build_state(xs, W, wl.H, wl.M, it, tile=wl.tile)
    for c in range(0, sample, wl.chunk):
        oracle.deslice(xs[c:c + wl.chunk], W["W2"], W["b2"], st["Z"], W["b3"], wl.H, wl.M, it)
    dt = time.perf_counter() - t0
    threads = max([p.get("num_threads", 1) for p in threadpool_info()] + [1])
    return {"value": sample / dt, "unit": "points/s", "cores": threads, "kind": "oracle",
            "sample": f"layer forward (pass 1, state, pass 2) in float64 numpy on the first {sample} "
                      f"points of the mesh: {dt:.1f} s"}


METRIC_BW = "mesh points/s per Physics-Attention layer fwd+bwd @2M pts C=128 fp32; % roofline"
PEAK_FP32_TFLOPS = 157.3    # MI355X dense float32 matrix peak


def cpu_baseline_backward(x_dev, g_dev, W, wl, sample):
    """The float64 oracle (as written): forward state and backward on the first
    `sample` points, host cores."""
    import numpy as np
    from threadpoolctl import threadpool_info

    from oracle import backward as BW
    xs = x_dev[:sample].double().cpu().numpy()
    gs = g_dev[:sample].double().cpu().numpy()
    W64 = {k: np.asarray(v, np.float64) for k, v in W.items()}
    t0 = time.perf_counter()
    BW.layer_backward(xs, W64, gs, wl.H, wl.M, 1.0 / wl.tau, tile=wl.tile)
    dt = time.perf_counter() - t0
    threads = max([p.get("num_threads", 1) for p in threadpool_info()] + [1])
    return {"value": sample / dt, "unit": "points/s", "cores": threads, "kind": "oracle",
            "sample": f"layer forward state + backward (all gradients) in float64 numpy on the first {sample} "
                      f"points of the mesh: {dt:.1f} s"}


def bench_backward(args):
    """A training step of one layer in float32: the forward over the resident
    points (which leaves the state the backward needs), then the backward with
    the slice weights recomputed tile by tile."""
    import torch

    from paper_2602_04940_amd import LayerWeights, PhysicsAttention
    from ts3_synth import WORKLOADS, make_weights
    from ts3_synth.device_gen import DeviceVolume

    wl = WORKLOADS["volume_2m_fp32"]
    N = args.points or wl.N
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    log(f"generating {N} volume points on the device (C={wl.C}, fp32) and an output gradient")
    x = torch.empty((N, wl.C), device=dev, dtype=torch.float32)
    DeviceVolume(wl.seed, wl.C, dev, dtype=torch.float32).fill(x)
    gen = torch.Generator(device=dev)
    gen.manual_seed(wl.seed + 1000)
    g = torch.randn((N, wl.C), device=dev, dtype=torch.float32, generator=gen)
    out = torch.empty_like(x)
    dx = torch.empty_like(x)
    W = make_weights(wl.C, wl.H, wl.M, wl.dh, seed=0)
    lw = LayerWeights(W, dev)
    layer = PhysicsAttention(wl.C, wl.H, wl.M, wl.dh, wl.tau, "fp32", group_span=wl.group_span, max_points=N)
    torch.cuda.synchronize()

    def step():
        layer.forward(lw, x, tile=wl.tile, chunk=wl.chunk, out=out)
        return layer.backward(lw, x, g, tile=wl.tile, dx=dx)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    log(f"warmup {args.warmup} done; timing {args.steps} steps")
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(args.steps):
        step()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / max(args.steps, 1)

    # forward and backward separately, on the launch stream
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
    reps = max(args.steps, 1)
    t_fw = t_bw = 0.0
    for _ in range(reps):
        ev[0].record()
        layer.forward(lw, x, tile=wl.tile, chunk=wl.chunk, out=out)
        ev[1].record()
        layer.backward(lw, x, g, tile=wl.tile, dx=dx)
        ev[2].record()
        torch.cuda.synchronize()
        t_fw += ev[0].elapsed_time(ev[1]) / reps
        t_bw += ev[1].elapsed_time(ev[2]) / reps
    log(f"{ms:.3f} ms/step: forward {t_fw:.3f} ms, backward {t_bw:.3f} ms")

    # algorithmic backward flops per point: logits recomputed (2), w^T g (2),
    # g.Z and x.ds_raw (4), x^T dz (2), dz W2^T (2), w ds_raw (2), each x C*H*M
    flop_bw = 14 * wl.C * wl.H * wl.M
    achieved = flop_bw * N / (t_bw * 1e-3) / 1e12
    roofline = {"bound": "mfma", "achieved": round(achieved, 2), "peak": PEAK_FP32_TFLOPS, "unit": "TFLOP/s",
                "frac": round(achieved / PEAK_FP32_TFLOPS, 4), "traffic": None,
                "kernel": "ts3_layer_backward (all launches)", "launch_ms": round(t_bw, 4), "launches": 1}
    result = {
        "metric": METRIC_BW, "value": N / (ms * 1e-3), "unit": "points/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": "synthetic: seeded volume mesh (box minus car-like body), Fourier features, device-generated; "
                "output gradient N(0,1)",
        "config": {"workload": wl.name, "N": N, "C": wl.C, "H": wl.H, "M": wl.M, "dh": wl.dh, "tau": wl.tau,
                   "tile": wl.tile, "chunk": wl.chunk, "group_span": wl.group_span},
        "passes_ms": {"forward": round(t_fw, 3), "backward": round(t_bw, 3)},
        "roofline": roofline,
        "cpu_baseline": None,
    }
    if not args.no_cpu_baseline:
        sample = min(args.cpu_sample_backward, N)
        log(f"timing the float64 backward oracle on {sample} points (host cores)")
        result["cpu_baseline"] = cpu_baseline_backward(x, g, W, wl, sample)
    layer.close()
    print(json.dumps(result), flush=True)


METRIC_STACK = "mesh points/s through an 8-block Transolver stack fwd @10M pts C=256 bf16; % roofline"
STACK_BLOCKS = 8


def cpu_baseline_stack(x_dev, blocks, wl, sample):
    """The float64 block oracle (as written) over the first `sample` points."""
    import numpy as np
    from threadpoolctl import threadpool_info

    from oracle import block as BK
    xs = x_dev[:sample].double().cpu().numpy()
    b64 = [{k: np.asarray(v, np.float64) for k, v in b.items()} for b in blocks]
    t0 = time.perf_counter()
    BK.stack_forward(xs, b64, wl.H, wl.M, 1.0 / wl.tau)
    dt = time.perf_counter() - t0
    threads = max([p.get("num_threads", 1) for p in threadpool_info()] + [1])
    return {"value": sample / dt, "unit": "points/s", "cores": threads, "kind": "oracle",
            "sample": f"{len(blocks)}-block stack forward in float64 numpy on the first {sample} points of the "
                      f"mesh (as their own mesh): {dt:.1f} s"}


def bench_stack(args):
    """The 8-block pre-norm Transolver stack (Physics-Attention + 4C feed-forward
    per block) over the 10M-point car surface, bf16 activations."""
    import torch

    from paper_2602_04940_amd import BlockWeights, PhysicsAttention, TransolverStack
    from ts3_synth import WORKLOADS, make_block_weights
    from ts3_synth.device_gen import DeviceSurface

    wl = WORKLOADS["car_10m_bf16"]
    N = args.points or wl.N
    F = 4 * wl.C
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    log(f"generating {N} car-surface points on the device (C={wl.C}, bf16)")
    x0 = torch.empty((N, wl.C), device=dev, dtype=torch.bfloat16)
    DeviceSurface(wl.seed, wl.C, dev).fill(x0)
    x = torch.empty_like(x0)
    blocks = [make_block_weights(wl.C, wl.H, wl.M, wl.dh, F, seed=100 + l) for l in range(STACK_BLOCKS)]
    dblocks = [BlockWeights(b, dev) for b in blocks]
    stack = TransolverStack(wl.C, wl.H, wl.M, STACK_BLOCKS, F, wl.dh, wl.tau, group_span=wl.group_span,
                            max_points=N)
    torch.cuda.synchronize()

    def step():
        stack.forward(dblocks, x, tile=wl.tile, chunk=wl.chunk)

    for _ in range(args.warmup):
        x.copy_(x0)
        step()
    torch.cuda.synchronize()
    log(f"warmup {args.warmup} done; timing {args.steps} steps (the input is restored between steps, untimed)")
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    total = 0.0
    for _ in range(args.steps):
        x.copy_(x0)
        torch.cuda.synchronize()
        e0.record()
        step()
        e1.record()
        torch.cuda.synchronize()
        total += e0.elapsed_time(e1)
    ms = total / max(args.steps, 1)
    log(f"{ms:.3f} ms/step")
    free, tot = torch.cuda.mem_get_info()

    # Per-kernel launch durations on the launch stream: one block's
    # Physics-Attention passes (a layer of the same shape) and its feed-forward.
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(5)]
    ntile, nchunk = -(-N // wl.tile), -(-N // wl.chunk)
    lw = dblocks[0].pa
    with PhysicsAttention(wl.C, wl.H, wl.M, wl.dh, wl.tau, "bf16", group_span=wl.group_span, max_points=N) as layer:
        pa = torch.empty_like(x0)
        layer.forward(lw, x0, tile=wl.tile, chunk=wl.chunk, out=pa)
        torch.cuda.synchronize()
        ev[0].record()
        layer.reset()
        for t in range(ntile):
            layer.accumulate(lw, x0[t * wl.tile:(t + 1) * wl.tile], t * wl.tile)
        ev[1].record()
        layer.finalize(lw)
        layer.attention(lw)
        ev[2].record()
        for c in range(nchunk):
            layer.deslice(lw, x0[c * wl.chunk:(c + 1) * wl.chunk], pa[c * wl.chunk:(c + 1) * wl.chunk])
        ev[3].record()
        torch.cuda.synchronize()
        x.copy_(x0)  # the feed-forward works in place; the copy is not timed
        ev5 = torch.cuda.Event(enable_timing=True)
        ev5.record()
        stack.feedforward(dblocks, 0, x, pa)
        ev[4].record()
        torch.cuda.synchronize()
    t_p1, t_mid, t_p2 = (ev[i].elapsed_time(ev[i + 1]) for i in range(3))
    t_ff = ev5.elapsed_time(ev[4])
    log(f"per block: pass1 {t_p1:.3f} ms ({ntile} launches), state {t_mid:.3f} ms, pass2 {t_p2:.3f} ms "
        f"({nchunk} launches), feed-forward {t_ff:.3f} ms (1 launch + fragment prep)")
    pa_flop = 4 * wl.C * wl.H * wl.M          # per point and pass
    ff_flop = 4 * wl.C * F                    # per point: two products of 2*C*F
    cands = [("k_mlp_residual", t_ff, 1, ff_flop * N), ("k_slice_accumulate_wide", t_p1, ntile, pa_flop * N),
             ("k_deslice", t_p2, nchunk, pa_flop * N)]
    kname, t_all, nl, flop_all = max(cands, key=lambda c: c[1])
    t_launch = t_all / nl
    achieved = flop_all / nl / (t_launch * 1e-3) / 1e12
    roofline = {"bound": "mfma", "achieved": round(achieved, 2), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                "frac": round(achieved / PEAK_BF16_TFLOPS, 4), "traffic": None, "kernel": kname,
                "launch_ms": round(t_launch, 4), "launches": nl}
    result = {
        "metric": METRIC_STACK, "value": N / (ms * 1e-3), "unit": "points/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic: seeded car-like surface mesh, Fourier features, device-generated; random-init blocks",
        "config": {"workload": wl.name, "N": N, "C": wl.C, "H": wl.H, "M": wl.M, "dh": wl.dh, "tau": wl.tau,
                   "blocks": STACK_BLOCKS, "hidden": F, "tile": wl.tile, "chunk": wl.chunk,
                   "group_span": wl.group_span, "hbm_used_gb": round((tot - free) / 1e9, 2)},
        "per_block_ms": {"pass1": round(t_p1, 3), "state": round(t_mid, 3), "pass2": round(t_p2, 3),
                         "feedforward": round(t_ff, 3)},
        "roofline": roofline,
        "cpu_baseline": None,
    }
    if not args.no_cpu_baseline:
        sample = min(args.cpu_sample_stack, N)
        log(f"timing the float64 stack oracle on {sample} points (host cores)")
        result["cpu_baseline"] = cpu_baseline_stack(x0, blocks, wl, sample)
    stack.close()
    print(json.dumps(result), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--points", type=int, default=None, help="override N (quick runs)")
    ap.add_argument("--cpu-sample", type=int, default=1_000_000)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--pmc-driver", action="store_true", help="short workload for rocprofv3 --pmc runs")
    ap.add_argument("--summarize-traffic", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="write profiles/traffic.json from two --pmc runs of --pmc-driver")
    ap.add_argument("--command", default="", help="command line recorded with --summarize-traffic")
    ap.add_argument("--backward", action="store_true",
                    help="time a float32 training step (forward + backward) on 2M points instead")
    ap.add_argument("--cpu-sample-backward", type=int, default=100_000)
    ap.add_argument("--stack", action="store_true",
                    help="time the 8-block Transolver stack on the 10M-point car surface (C=256) instead")
    ap.add_argument("--cpu-sample-stack", type=int, default=20_000)
    ap.add_argument("--accum", choices=("fp32", "fp64"), default="fp32",
                    help="precision of the fold of span partials (float64: Appendix A.4 robustness)")
    args = ap.parse_args()
    if args.summarize_traffic:
        summarize_traffic(*args.summarize_traffic, args.command)
        return
    if args.pmc_driver:
        pmc_driver(args.points or 4_000_000)
        return
    if args.gpus != 1:
        print(f"bench.py: this build measures one GPU; --gpus {args.gpus} is not supported "
              "(the layer shards by points with one all-gather of span partials; not built here)",
              file=sys.stderr)
        sys.exit(2)
    if args.backward:
        bench_backward(args)
        return
    if args.stack:
        bench_stack(args)
        return

    import numpy as np
    import torch

    from paper_2602_04940_amd import LayerWeights, PhysicsAttention
    from ts3_synth import WORKLOADS, make_weights
    from ts3_synth.device_gen import DeviceVolume

    wl = WORKLOADS["volume_100m_bf16"]
    N = args.points or wl.N
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    log(f"generating {N} volume points on the device (C={wl.C}, bf16)")
    t0 = time.perf_counter()
    x = torch.empty((N, wl.C), device=dev, dtype=torch.bfloat16)
    DeviceVolume(wl.seed, wl.C, dev).fill(x, progress=lambda k: log(f"  chunk {k}/{-(-N // 1_000_000)}"))
    out = torch.empty_like(x)
    torch.cuda.synchronize()
    log(f"inputs ready in {time.perf_counter() - t0:.1f} s")

    W = make_weights(wl.C, wl.H, wl.M, wl.dh, seed=0)
    lw = LayerWeights(W, dev)
    layer = PhysicsAttention(wl.C, wl.H, wl.M, wl.dh, wl.tau, "bf16", group_span=wl.group_span, max_points=N,
                             accum=args.accum)
    free, total = torch.cuda.mem_get_info()
    hbm_used_gb = (total - free) / 1e9

    for i in range(args.warmup):
        layer.forward(lw, x, tile=wl.tile, chunk=wl.chunk, out=out)
    torch.cuda.synchronize()
    log(f"warmup {args.warmup} done; timing {args.steps} steps")

    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for i in range(args.steps):
        layer.forward(lw, x, tile=wl.tile, chunk=wl.chunk, out=out)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / max(args.steps, 1)
    log(f"{ms:.3f} ms/step")

    # Per-pass launch durations on the launch stream (torch's current stream).
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
    ntile = -(-N // wl.tile)
    nchunk = -(-N // wl.chunk)
    ev[0].record()
    layer.reset()
    for t in range(ntile):
        layer.accumulate(lw, x[t * wl.tile:(t + 1) * wl.tile], t * wl.tile)
    ev[1].record()
    layer.finalize(lw)
    layer.attention(lw)
    ev[2].record()
    for c in range(nchunk):
        layer.deslice(lw, x[c * wl.chunk:(c + 1) * wl.chunk], out[c * wl.chunk:(c + 1) * wl.chunk])
    ev[3].record()
    torch.cuda.synchronize()
    t_p1, t_mid, t_p2 = (ev[i].elapsed_time(ev[i + 1]) for i in range(3))
    log(f"pass1 {t_p1:.3f} ms ({ntile} launches), state {t_mid:.3f} ms, pass2 {t_p2:.3f} ms ({nchunk} launches)")

    flop_per_point = 4 * wl.C * wl.H * wl.M        # logits + contraction, per pass
    if t_p1 >= t_p2:
        kname, t_launch, nl = "k_slice_accumulate_pc", t_p1 / ntile, ntile
    else:
        kname, t_launch, nl = "k_deslice_w8", t_p2 / nchunk, nchunk
    pts_launch = min(wl.tile, N)
    achieved = flop_per_point * pts_launch / (t_launch * 1e-3) / 1e12
    traffic = measured_traffic(kname, pts_launch)
    roofline = {"bound": "mfma", "achieved": round(achieved, 2), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                "frac": round(achieved / PEAK_BF16_TFLOPS, 4), "traffic": traffic, "kernel": kname,
                "launch_ms": round(t_launch, 4), "launches": nl}

    result = {
        "metric": METRIC, "value": N / (ms * 1e-3), "unit": "points/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic: seeded volume mesh (box minus car-like body), Fourier features, device-generated",
        "config": {"workload": wl.name, "N": N, "C": wl.C, "H": wl.H, "M": wl.M, "dh": wl.dh, "tau": wl.tau,
                   "tile": wl.tile, "chunk": wl.chunk, "group_span": wl.group_span, "accum": args.accum,
                   "hbm_used_gb": round(hbm_used_gb, 2), "state_bytes": layer.bytes()},
        "passes_ms": {"pass1": round(t_p1, 3), "state": round(t_mid, 3), "pass2": round(t_p2, 3)},
        "roofline": roofline,
        "cpu_baseline": None,
    }
    if not args.no_cpu_baseline:
        log(f"timing the float64 oracle on {args.cpu_sample} points (host cores)")
        result["cpu_baseline"] = cpu_baseline(x, W, wl, min(args.cpu_sample, N))
    layer.close()
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
