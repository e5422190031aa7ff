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
drawn by seed without replacement from a 160M-point volume mesh (C=128, H=8,
M=64, 1M-point tiles), with the backward's roofline against the float32 matrix
peak and the float64 backward oracle as the CPU baseline.

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


def pmc_driver(points: int, workloads=("layer",)):
    """Short workload for rocprofv3 --pmc runs.  "layer": two layer forwards over
    `points` points of the 100M-point volume mesh's recipe (1M-point launches);
    "stack": one block's feed-forward and both passes at C=256 on 1M car-surface
    points; "backward": a float32 forward and backward on 1M volume points.
    Ends with one device-to-device copy of CAL_BYTES whose counter readings
    calibrate FETCH_SIZE / WRITE_SIZE."""
    import torch

    from paper_2602_04940_amd import BlockWeights, LayerWeights, PhysicsAttention, TransolverStack
    from ts3_synth import WORKLOADS, make_block_weights, make_weights
    from ts3_synth.device_gen import DeviceSurface, DeviceVolume
    if "layer" in workloads:
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
        del x, out
        log("pmc driver: layer done")
    if "stack" in workloads:
        wl = WORKLOADS["car_10m_bf16"]
        n, F = 1_000_000, 4 * wl.C
        x = torch.empty((n, wl.C), device="cuda", dtype=torch.bfloat16)
        DeviceSurface(wl.seed, wl.C).fill(x)
        blocks = [BlockWeights(make_block_weights(wl.C, wl.H, wl.M, wl.dh, F, seed=100 + l)) for l in range(2)]
        stack = TransolverStack(wl.C, wl.H, wl.M, 2, F, wl.dh, wl.tau, group_span=wl.group_span, max_points=n)
        stack.forward(blocks, x, tile=wl.tile, chunk=wl.chunk)
        torch.cuda.synchronize()
        stack.close()
        del x
        log("pmc driver: stack done")
    if "backward" in workloads:
        from ts3_synth.workloads import subset_indices
        wl = WORKLOADS["volume_2m_fp32"]
        n = 1_000_000
        x = torch.empty((n, wl.C), device="cuda", dtype=torch.float32)
        DeviceVolume(wl.seed, wl.C, dtype=torch.float32).gather(x, subset_indices(wl)[:n], wl.source_N)
        gen = torch.Generator(device="cuda")
        gen.manual_seed(wl.seed + 1000)
        g = torch.randn((n, wl.C), device="cuda", dtype=torch.float32, generator=gen)
        lw = LayerWeights(make_weights(wl.C, wl.H, wl.M, wl.dh, seed=0))
        with PhysicsAttention(wl.C, wl.H, wl.M, wl.dh, wl.tau, "fp32", group_span=wl.group_span,
                              max_points=n) as layer:
            layer.forward(lw, x, tile=wl.tile, chunk=wl.chunk)
            layer.backward(lw, x, g, tile=wl.tile)
            torch.cuda.synchronize()
        del x, g
        log("pmc driver: backward done")
    src = torch.empty(CAL_BYTES, device="cuda", dtype=torch.uint8).fill_(1)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    dst.copy_(src)
    torch.cuda.synchronize()
    log("pmc driver done")


# Kernels whose counters are summarised: name prefix -> (points per dispatch,
# matrix flop per point that the kernel executes, algorithmic HBM bytes per
# point, peak TFLOP/s of its matrix dtype).  The first forward kernels execute
# 4*C*H*M (logits and one contraction).  The projected pass 1 executes
# 2*(C*H*M + 2*C*C + 4*M*C): logits, x W1 per head (rounded W1 and its
# remainder), the weighted sums of the projected rows (rounded value and
# remainder), their weight sums and the softmax row sums; the slice-state
# pass 2 executes 2*(C*H*M + 2*M*C + C*C): logits, w s' per head, the row
# sums, and Linear3.  The backward's dZ kernel 4, its dx kernel 10 and its dW2
# kernel 2 (x C*H*M), of which the backward as a whole needs 14.  The dx
# kernel writes dz (H*M floats per point), which the dW2 kernel reads.
SQ_COUNTERS = ("SQ_INSTS_MFMA SQ_VALU_MFMA_BUSY_CYCLES SQ_INSTS_VALU SQ_INSTS_VALU_TRANS_F32 "
               "SQ_INSTS_LDS SQ_LDS_BANK_CONFLICT SQ_LDS_IDX_ACTIVE SQ_BUSY_CYCLES GRBM_GUI_ACTIVE")
COUNTER_KERNELS = {
    "k_slice_accumulate_pc<": (1_000_000, 4 * 128 * 512, 256, PEAK_BF16_TFLOPS),
    "k_deslice_w8<": (1_000_000, 4 * 128 * 512, 512, PEAK_BF16_TFLOPS),
    "k_slice_accumulate_pcp<": (1_000_000, 2 * (128 * 512 + 2 * 128 * 128 + 4 * 64 * 128), 256, PEAK_BF16_TFLOPS),
    "k_deslice_sf<": (1_000_000, 2 * (128 * 512 + 2 * 64 * 128 + 128 * 128), 512, PEAK_BF16_TFLOPS),
    "k_slice_accumulate_pcw<": (1_000_000, 4 * 256 * 512, 512, PEAK_BF16_TFLOPS),
    "k_deslice_pc<": (1_000_000, 4 * 256 * 512, 1024, PEAK_BF16_TFLOPS),
    "k_mlp_residual_pc<": (1_000_000, 4 * 256 * 1024, 1536, PEAK_BF16_TFLOPS),
    "k_bw_head<": (1_000_000, 4 * 128 * 512, 1024, 157.3),
    "k_bw_dx<": (1_000_000, 10 * 128 * 512, 1536 + 4 * 512, 157.3),
    "k_bw_dw2<": (1_000_000, 2 * 128 * 512, 512 + 4 * 512, 157.3),
}


def summarize_counters(sq_dir: str, fetch_dir: str, write_dir: str, command: str, out_path: str):
    """Per-kernel counter summary (text) from three rocprofv3 runs of --pmc-driver:
    the SQ/GRBM counters with --kernel-trace, then FETCH_SIZE, then WRITE_SIZE."""
    import csv
    import glob

    def rows(d, pattern):
        f = glob.glob(os.path.join(d, "**", pattern), recursive=True)
        if not f:
            raise SystemExit(f"no {pattern} under {d}")
        return list(csv.DictReader(open(f[0])))

    def per_kernel(rs, name):
        acc = {}
        for r in rs:
            if r["Counter_Name"] != name:
                continue
            for k in COUNTER_KERNELS:
                if k in r["Kernel_Name"]:
                    acc.setdefault(k, []).append(float(r["Counter_Value"]))
        return {k: sum(v) / len(v) for k, v in acc.items()}, {k: len(v) for k, v in acc.items()}

    sq = rows(sq_dir, "*counter_collection.csv")
    # GRBM_GUI_ACTIVE comes summed over the XCDs; the SQ counters over every
    # CU and SIMD.  Shapes from the agent table of the same run.
    gpu = [a for a in rows(sq_dir, "*agent_info.csv") if int(a.get("Simd_Count", 0) or 0) > 0][0]
    n_xcc, n_cu, n_simd = int(gpu["Num_Xcc"]), int(gpu["Cu_Count"]), int(gpu["Simd_Count"])
    trace = rows(sq_dir, "*kernel_trace.csv")
    dur = {}
    for r in trace:
        for k in COUNTER_KERNELS:
            if k in r["Kernel_Name"]:
                dur.setdefault(k, []).append((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-9)
    vals = {}
    ndisp = {}
    for name in SQ_COUNTERS.split():
        v, n = per_kernel(sq, name)
        vals[name] = v
        ndisp.update(n)
    fac = {}
    for name, d in (("FETCH_SIZE", fetch_dir), ("WRITE_SIZE", write_dir)):
        rs = rows(d, "*counter_collection.csv")
        cal = [r for r in rs if r["Counter_Name"] == name and "copyBuffer" in r["Kernel_Name"]][-1]
        fac[name] = CAL_BYTES / (float(cal["Counter_Value"]) * 1024.0)
        vals[name] = per_kernel(rs, name)[0]
    lines = [f"rocprofv3 counters per dispatch (averages over the dispatches of each kernel), one MI355X",
             f"command: {command}",
             f"calibration: FETCH_SIZE x{fac['FETCH_SIZE']:.4f}, WRITE_SIZE x{fac['WRITE_SIZE']:.4f} bytes per "
             f"counted byte (a {CAL_BYTES >> 20} MiB device-to-device copy)",
             "duration: kernel-trace average of the SQ run (counter collection serialises dispatches)",
             f"GPU: {n_xcc} XCDs, {n_cu} CUs, {n_simd} SIMDs; cycles = GRBM_GUI_ACTIVE / {n_xcc} (the counter is summed "
             "over the XCDs); clock = cycles / duration;",
             "mfma%: SQ_VALU_MFMA_BUSY_CYCLES / (cycles x SIMDs); lds%: SQ_LDS_IDX_ACTIVE / (cycles x CUs); "
             "bank%: SQ_LDS_BANK_CONFLICT / (cycles x CUs);",
             "frac: executed matrix flop / duration / the dtype's dense peak; HBM: FETCH_SIZE + WRITE_SIZE, calibrated",
             ""]
    hdr = (f"{'kernel':26s} {'disp':>4s} {'us':>8s} {'GHz':>5s} {'TF/s':>7s} {'frac':>6s} {'mfma%':>6s} "
           f"{'VALU/MFMA':>9s} {'TRANS/MFMA':>10s} {'LDS/MFMA':>8s} {'lds%':>5s} {'bank%':>6s} {'HBM MB':>8s} "
           f"{'algo MB':>8s} {'GB/s':>7s}")
    lines.append(hdr)
    out = {}
    for k, (pts, flop_pt, bytes_pt, peak) in COUNTER_KERNELS.items():
        if k not in dur or k not in vals["SQ_INSTS_MFMA"]:
            continue
        t = sum(dur[k]) / len(dur[k])
        g = vals["GRBM_GUI_ACTIVE"].get(k, float("nan")) / n_xcc
        mf = vals["SQ_INSTS_MFMA"][k]
        busy = vals["SQ_VALU_MFMA_BUSY_CYCLES"].get(k, float("nan"))
        hbm = (vals["FETCH_SIZE"].get(k, float("nan")) * fac["FETCH_SIZE"] +
               vals["WRITE_SIZE"].get(k, float("nan")) * fac["WRITE_SIZE"]) * 1024
        tf = flop_pt * pts / t / 1e12
        row = {"dispatches": ndisp.get(k), "us": t * 1e6, "clock_ghz": g / t / 1e9, "tflops": tf,
               "frac": tf / peak, "mfma_busy": busy / (g * n_simd) if g else None,
               "valu_per_mfma": vals["SQ_INSTS_VALU"][k] / mf, "trans_per_mfma":
               vals["SQ_INSTS_VALU_TRANS_F32"][k] / mf, "lds_per_mfma": vals["SQ_INSTS_LDS"][k] / mf,
               "lds_busy": vals["SQ_LDS_IDX_ACTIVE"][k] / (g * n_cu) if g else None,
               "bank_conflict": vals["SQ_LDS_BANK_CONFLICT"][k] / (g * n_cu) if g else None,
               "hbm_mb": hbm / 1e6, "algo_mb": bytes_pt * pts / 1e6, "gbs": hbm / t / 1e9}
        out[k] = row
        lines.append(f"{k.rstrip('<'):26s} {row['dispatches']:4d} {row['us']:8.1f} {row['clock_ghz']:5.2f} "
                     f"{tf:7.1f} {row['frac']:6.3f} {100 * row['mfma_busy']:6.1f} {row['valu_per_mfma']:9.2f} "
                     f"{row['trans_per_mfma']:10.2f} {row['lds_per_mfma']:8.2f} {100 * row['lds_busy']:5.1f} "
                     f"{100 * row['bank_conflict']:6.2f} "
                     f"{row['hbm_mb']:8.1f} {row['algo_mb']:8.1f} {row['gbs']:7.0f}")
    lines += ["", f"kernel source hash {kernel_source_hash()}"]
    text = "\n".join(lines) + "\n"
    os.makedirs(os.path.dirname(out_path) or ".", exist_ok=True)
    with open(out_path, "w") as fh:
        fh.write(text)
    print(text)
    return out


def summarize_trace(trace_dir: str, command: str, out_path: str, title: str):
    """Kernel-trace summary (text) of one rocprofv3 --kernel-trace run: every
    kernel's calls and durations, and separately the launches that overlapped
    no other launch of this library (single-stream launch durations)."""
    import csv
    import glob

    f = glob.glob(os.path.join(trace_dir, "**", "*kernel_trace.csv"), recursive=True)
    if not f:
        raise SystemExit(f"no kernel_trace.csv under {trace_dir}")
    rows = [r for r in csv.DictReader(open(f[0])) if "ts3::" in r["Kernel_Name"]]
    ev = sorted((int(r["Start_Timestamp"]), int(r["End_Timestamp"]), r["Kernel_Name"]) for r in rows)

    def table(items):
        agg = {}
        for a, b, k in items:
            agg.setdefault(k, []).append((b - a) * 1e-3)
        out = [f"{'kernel':62s} {'calls':>6s} {'avg_us':>10s} {'min_us':>10s} {'max_us':>10s}"]
        for k, v in sorted(agg.items(), key=lambda kv: -sum(kv[1])):
            out.append(f"{k[:62]:62s} {len(v):6d} {sum(v) / len(v):10.1f} {min(v):10.1f} {max(v):10.1f}")
        return out

    alone = []
    for i, (a, b, k) in enumerate(ev):
        prev_end = max((e[1] for e in ev[max(0, i - 8):i]), default=0)
        nxt = ev[i + 1][0] if i + 1 < len(ev) else b + 1
        if a >= prev_end and nxt >= b:
            alone.append((a, b, k))
    lines = [title, f"command: {command}", "", "All launches:"] + table(ev)
    lines += ["", "Launches that overlapped no other launch of the library:"] + table(alone)
    lines += ["", f"kernel source hash {kernel_source_hash()}"]
    text = "\n".join(lines) + "\n"
    os.makedirs(os.path.dirname(out_path) or ".", exist_ok=True)
    with open(out_path, "w") as fh:
        fh.write(text)
    print(text)


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
        for kname in ("k_slice_accumulate_pc", "k_slice_accumulate_pcp", "k_deslice_w8", "k_deslice_sf"):
            vals = [float(r["Counter_Value"]) for r in rs if kname + "<" in r["Kernel_Name"]]
            if vals:  # kernels the workload did not run are left out
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


def cpu_baseline_and_parity(x_dev, W, lw, wl, sample):
    """The float64 oracle (as written) on the first `sample` points of the mesh,
    taken as a mesh of its own, on a pool of host processes (one core each):
    pass 1 over 65,536-point tiles summed in tile order, the token side, pass 2
    over 65,536-point chunks.  Then the GPU layer runs the same sample with the
    benchmark's launch configuration, and its state and output are compared
    with the oracle's: the parity of this run."""
    import numpy as np

    from oracle.pool import OraclePool
    from paper_2602_04940_amd import PhysicsAttention, _lib as L
    xs = x_dev[:sample]
    x64 = xs.float().cpu().numpy().astype(np.float64)
    it = 1.0 / wl.tau
    with OraclePool() as pool:
        pool.sums([x64[:64]], W["W2"], W["b2"], wl.H, wl.M, it)  # workers started before the clock
        t0 = time.perf_counter()
        st = pool.state(x64, W, wl.H, wl.M, it, tile=65536)
        ref = pool.decode(x64, W["W2"], W["b2"], st["Z"], W["b3"], wl.H, wl.M, it, chunk=65536)
        dt = time.perf_counter() - t0
        workers = pool.workers
    base = {"value": sample / dt, "unit": "points/s", "cores": workers, "kind": "oracle",
            "sample": f"layer forward (pass 1, state, pass 2) in float64 numpy on the first {sample} points of "
                      f"the mesh as their own mesh, {workers} processes of one core each: {dt:.1f} s"}
    import torch
    with PhysicsAttention(wl.C, wl.H, wl.M, wl.dh, wl.tau, "bf16", group_span=wl.group_span,
                          max_points=sample) as layer:
        out = layer.forward(lw, xs, tile=wl.tile, chunk=wl.chunk)
        torch.cuda.synchronize()
        proj = layer.projected()
        g_sr, g_d, g_z = layer.get(L.TS3_T_RAW if proj else L.TS3_S_RAW), layer.get(L.TS3_D), layer.get(L.TS3_ZP)
    if proj:  # the state keeps sums of projected rows: compare with the oracle's
        with OraclePool() as pool:
            parts = pool.projected_tile_sums(x64, W["W2"], W["b2"], W["W1"], wl.H, wl.M, it, 65536)
        ref_sums = sum((t[0] for t in parts), np.zeros((wl.H, wl.M, wl.dh)))
    else:
        ref_sums = st["s_raw"]
    got = out.float().cpu().numpy().astype(np.float64)

    def rel(a, b):
        return float(np.linalg.norm(a - b) / np.linalg.norm(b))

    nb = sample // 256
    d2 = ((got[:nb * 256] - ref[:nb * 256]) ** 2).sum(axis=1).reshape(nb, 256).sum(axis=1)
    r2 = (ref[:nb * 256] ** 2).sum(axis=1).reshape(nb, 256).sum(axis=1)
    rn = np.linalg.norm(ref, axis=1)
    row = np.linalg.norm(got - ref, axis=1) / np.maximum(rn, np.sqrt((rn ** 2).mean()))
    HM = wl.H * wl.M
    tok = np.linalg.norm((g_sr - ref_sums).reshape(HM, -1), axis=1) / np.linalg.norm(
        ref_sums.reshape(HM, -1), axis=1)
    parity = {"sample": f"first {sample} points as their own mesh, group span {wl.group_span}, "
                        f"{wl.tile}-point tiles and chunks",
              "bar": 0.02, "out_rel_l2": rel(got, ref), "out_worst_256_block": float(np.sqrt(d2 / r2).max()),
              "out_worst_row": float(row.max()), ("t_raw" if proj else "s_raw") + "_worst_token": float(tok.max()),
              "d_worst_rel": float((np.abs(g_d - st["d"]) / st["d"]).max()), "Z_rel_l2": rel(g_z, st["Z"])}
    parity["pass"] = all(v <= 0.02 for k, v in parity.items() if k not in ("sample", "bar"))
    return base, parity


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
    threads = min(max([p.get("num_threads", 1) for p in threadpool_info()] + [1]), len(os.sched_getaffinity(0)))
    return {"value": sample / dt, "unit": "points/s", "cores": threads, "kind": "oracle",
            "sample": f"layer forward state + backward (all gradients) in float64 numpy on the first {sample} "
                      f"points of the training subset: {dt:.1f} s"}


def bench_backward(args):
    """A training step of one layer in float32: the forward over the resident
    points (which leaves the state the backward needs), then the backward with
    the slice weights recomputed tile by tile."""
    import torch

    from paper_2602_04940_amd import LayerWeights, PhysicsAttention
    from ts3_synth import WORKLOADS, make_weights
    from ts3_synth.device_gen import DeviceVolume

    from ts3_synth.workloads import subset_indices
    wl = WORKLOADS["volume_2m_fp32"]
    N = args.points or wl.N
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    log(f"drawing {N} of the {wl.source_N} points of the volume mesh (seed {wl.subset_seed}) on the device "
        f"(C={wl.C}, fp32), and an output gradient")
    x = torch.empty((N, wl.C), device=dev, dtype=torch.float32)
    DeviceVolume(wl.seed, wl.C, dev, dtype=torch.float32).gather(
        x, subset_indices(wl)[:N], wl.source_N, progress=lambda k: log(f"  mesh chunk {k}/{wl.source_N // 1_000_000}"))
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
        "data": f"synthetic: {N} points drawn uniformly without replacement (seed {wl.subset_seed}) from a "
                f"{wl.source_N}-point seeded volume mesh (box minus car-like body), Fourier features, "
                "device-generated; output gradient N(0,1)",
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
    threads = min(max([p.get("num_threads", 1) for p in threadpool_info()] + [1]), len(os.sched_getaffinity(0)))
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
    cands = [("k_mlp_residual_pc", t_ff, 1, ff_flop * N), ("k_slice_accumulate_pcw", t_p1, ntile, pa_flop * N),
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
    ap.add_argument("--cpu-sample", type=int, default=2_000_000)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--pmc-driver", action="store_true", help="short workload for rocprofv3 --pmc runs")
    ap.add_argument("--pmc-workloads", default="layer",
                    help="comma list of layer,stack,backward for --pmc-driver")
    ap.add_argument("--summarize-counters", nargs=4, metavar=("SQ_DIR", "FETCH_DIR", "WRITE_DIR", "OUT"),
                    help="per-kernel counter summary from three rocprofv3 runs of --pmc-driver")
    ap.add_argument("--summarize-traffic", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="write profiles/traffic.json from two --pmc runs of --pmc-driver")
    ap.add_argument("--command", default="", help="command line recorded with --summarize-traffic")
    ap.add_argument("--summarize-trace", nargs=3, metavar=("TRACE_DIR", "OUT", "TITLE"),
                    help="kernel-trace summary of a rocprofv3 --kernel-trace run")
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
    if args.summarize_trace:
        summarize_trace(args.summarize_trace[0], args.command, args.summarize_trace[1], args.summarize_trace[2])
        return
    if args.summarize_counters:
        summarize_counters(*args.summarize_counters[:3], args.command, args.summarize_counters[3])
        return
    if args.pmc_driver:
        pmc_driver(args.points or 4_000_000, tuple(args.pmc_workloads.split(",")))
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
    torch.cuda.synchronize()
    torch.cuda.empty_cache()  # drop the generator's cached blocks: what remains is x, out and the state
    free, total = torch.cuda.mem_get_info()
    hbm_used_gb = (total - free) / 1e9
    layer_bytes = 2 * x.numel() * x.element_size() + layer.bytes()

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

    # Algorithmic flop per point and pass (Table 2's N-terms): the logits
    # 2*C*H*M and one contraction with the slices 2*H*M*C.  The kernels reach
    # the same result with fewer products by reassociating the linear steps
    # (projected pass 1, slice-state pass 2); what they execute is reported
    # beside it.
    C, H, M = wl.C, wl.H, wl.M
    flop_per_point = 4 * C * H * M
    proj = layer.projected()
    sf = H * 16 == C  # the slice-state pass 2 serves head width 16
    p1 = ("k_slice_accumulate_pcp", 2 * (C * H * M + 2 * C * C + 4 * M * C)) if proj else \
        ("k_slice_accumulate_pc", flop_per_point)
    p2 = ("k_deslice_sf", 2 * (C * H * M + 2 * M * C + C * C)) if sf else ("k_deslice_w8", flop_per_point)
    if t_p1 >= t_p2:
        (kname, exec_pt), t_launch, nl = p1, t_p1 / ntile, ntile
    else:
        (kname, exec_pt), t_launch, nl = p2, t_p2 / nchunk, nchunk
    pts_launch = min(wl.tile, N)
    achieved = flop_per_point * pts_launch / (t_launch * 1e-3) / 1e12
    executed = exec_pt * pts_launch / (t_launch * 1e-3) / 1e12
    traffic = measured_traffic(kname, pts_launch)
    layer_tflops = 2 * flop_per_point * N / (ms * 1e-3) / 1e12   # both passes over the timed step
    layer_exec = (p1[1] + p2[1]) * N / (ms * 1e-3) / 1e12
    roofline = {"bound": "mfma", "achieved": round(achieved, 2), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                "frac": round(achieved / PEAK_BF16_TFLOPS, 4), "traffic": traffic, "kernel": kname,
                "launch_ms": round(t_launch, 4), "launches": nl,
                "executed_achieved": round(executed, 2), "executed_frac": round(executed / PEAK_BF16_TFLOPS, 4),
                "executed_flop_per_point": exec_pt, "algorithmic_flop_per_point": flop_per_point,
                "layer_achieved": round(layer_tflops, 2), "layer_frac": round(layer_tflops / PEAK_BF16_TFLOPS, 4),
                "layer_executed_frac": round(layer_exec / PEAK_BF16_TFLOPS, 4)}

    result = {
        "metric": METRIC, "value": N / (ms * 1e-3), "unit": "points/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic: seeded volume mesh (box minus car-like body), Fourier features, device-generated",
        "config": {"workload": wl.name, "N": N, "C": wl.C, "H": wl.H, "M": wl.M, "dh": wl.dh, "tau": wl.tau,
                   "tile": wl.tile, "chunk": wl.chunk, "group_span": wl.group_span, "accum": args.accum,
                   "hbm_used_gb": round(hbm_used_gb, 2), "hbm_layer_gb": round(layer_bytes / 1e9, 2),
                   "state_bytes": layer.bytes()},
        "passes_ms": {"pass1": round(t_p1, 3), "state": round(t_mid, 3), "pass2": round(t_p2, 3)},
        "roofline": roofline,
        "cpu_baseline": None,
        "parity": None,
    }
    layer.close()
    if not args.no_cpu_baseline:
        log(f"timing the float64 oracle on {args.cpu_sample} points (host processes), then parity on them")
        result["cpu_baseline"], result["parity"] = cpu_baseline_and_parity(x, W, lw, wl, min(args.cpu_sample, N))
        log(f"parity: {result['parity']}")
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
