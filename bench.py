"""Benchmark: DONeRF per-ray inference, 400x400 frames, N = 4, bf16 networks.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]
                    [--cpu-sample RAYS | --no-cpu]

One step renders the workload's 5 seeded poses (5 x 400 x 400 = 800,000 rays)
with one donerf_render call (one kernel launch) on inputs already resident:
weights on the device since donerf_create, poses passed by value.  Prints one
JSON line.  The roofline object is for the fused render kernel; its time is
measured with HIP events on the stream the kernel runs on.  The CPU baseline
is the oracle (bf16-rounding mode) timed on a seeded sample of the same rays.
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

MFMA_PEAK_TFLOPS = {"bf16": 2500.0, "fp32": 157.3, "fp8": 5000.0}   # MI355X dense peaks
HBM_PEAK_GBS = 8000.0

# HBM KiB per dispatch from two rocprofv3 --pmc runs (FETCH_SIZE, then
# WRITE_SIZE; profiles/*_traffic.md) scaled by the same counters on a plain
# 256 MiB copy (FETCH_SIZE reads half the bytes moved: x2; WRITE_SIZE exact:
# x1), per workload, valid only for the kernel sources they were taken with.
MEASURED_TRAFFIC = {
    "frame400_n4_bf16": {"sources_sha256_16": "592a453b4efe06fb", "fetch_kib": 7307.0 * 2, "write_kib": 11760.0},
    "targets400_b128_k5_z5": {"sources_sha256_16": "80e10b6e7a011a43", "fetch_kib": 9065.9 * 2, "write_kib": 400000.0},
}
# the sources (and the build script, whose flags shape the code) each
# measured kernel is built from
KERNEL_SOURCES = {
    "frame400_n4_bf16": ("paper_2103_03231_amd/csrc/render_kernel.h", "paper_2103_03231_amd/csrc/render_bf16_topn.hip",
                         "paper_2103_03231_amd/csrc/layout.h", "paper_2103_03231_amd/csrc/internal.h",
                         "paper_2103_03231_amd/build.py"),
    "targets400_b128_k5_z5": ("paper_2103_03231_amd/csrc/targets.hip", "paper_2103_03231_amd/csrc/internal.h",
                              "paper_2103_03231_amd/build.py"),
    "stereo1440x1600_n16_b256_cdf_bf16": ("paper_2103_03231_amd/csrc/render_kernel.h",
                                          "paper_2103_03231_amd/csrc/render_bf16_cdf_wide.hip",
                                          "paper_2103_03231_amd/csrc/layout.h", "paper_2103_03231_amd/csrc/internal.h",
                                          "paper_2103_03231_amd/build.py"),
}


def measured_traffic(workload):
    """HBM bytes per dispatch if counters were taken for the current sources."""
    m = MEASURED_TRAFFIC.get(workload)
    if m is None or m["sources_sha256_16"] != kernel_sources_sha(workload):
        return None
    return round((m["fetch_kib"] + m["write_kib"]) * 1024)


def kernel_sources_sha(workload: str = "frame400_n4_bf16") -> str:
    import hashlib
    h = hashlib.sha256()
    for f in KERNEL_SOURCES[workload]:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def depth_in_folded(depth_input: str) -> int:
    """Inputs of the first depth layer as evaluated: 90 encoded values, or the
    9 columns the unencoded positions input folds into (its 6 + 3 B inputs
    are affine in the ray)."""
    return {"encoded": 90, "positions": 9}[depth_input]


def algorithmic_flop_per_ray(N: int, n_bins: int, d_in: int = 90) -> int:
    """2 x multiply-adds of both networks for one ray (8 layers of 256 units):
    depth network d_in->256, 6 x 256->256, 256->B once; shading network
    63->256, 6 x 256->256, 283->4 for each of the N samples."""
    d = d_in * 256 + 6 * 256 * 256 + 256 * n_bins
    s = 63 * 256 + 6 * 256 * 256 + (256 + 27) * 4
    return 2 * (d + N * s)


def fp8_flop_per_ray(N: int) -> int:
    """The part of the algorithmic work the mixed fp8 network runs in fp8:
    the six 256 -> 256 hidden layers of both networks."""
    return 2 * 6 * 256 * 256 * (1 + N)


def mixed_peak(N: int, n_bins: int, d_in: int) -> float:
    """Peak of the mixed fp8 network: the time its work takes at the fp8 and
    bf16 dense peaks, each part at its own."""
    tot = algorithmic_flop_per_ray(N, n_bins, d_in)
    f8 = fp8_flop_per_ray(N)
    t = f8 / MFMA_PEAK_TFLOPS["fp8"] + (tot - f8) / MFMA_PEAK_TFLOPS["bf16"]
    return tot / t


def padded_flop_per_ray(N: int, n_bins: int, d_in: int = 90, head_sweeps: int = 1) -> int:
    """2 x multiply-adds the MFMA tiles execute (K padded to 96 (16 for the
    folded positions layer) / 64 / 288, shading head padded to 32 rows; the
    depth head twice where inverse-CDF placement over more than 128 classes
    runs it in two sweeps)."""
    d = (96 if d_in == 90 else 16) * 256 + 6 * 256 * 256 + head_sweeps * 256 * n_bins
    s = 64 * 256 + 6 * 256 * 256 + 288 * 32
    return 2 * (d + N * s)


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def cpu_baseline(wl, weights, poses, n_sample):
    """The oracle on a seeded uniform sample of the workload's rays, timed on
    this host; rays/s and the time per frame extrapolated from the sample."""
    from threadpoolctl import threadpool_info

    from oracle import donerf_oracle as O
    rng = np.random.default_rng(1234)
    total = wl.rays
    sub = np.sort(rng.choice(total, size=min(n_sample, total), replace=False))
    log(f"cpu baseline: oracle ({wl.precision}) on {len(sub)} sampled rays")
    t0 = time.perf_counter()
    O.render(weights, poses, wl.H, wl.W, wl.N, n_bins=wl.n_bins, fov_x_deg=wl.fov_deg,
             precision=wl.precision, select=wl.select, ray_subset=sub, depth_input=wl.depth_input)
    dt = time.perf_counter() - t0
    threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    rate = len(sub) / dt
    return {"value": rate / 1e6, "unit": "Mrays/s", "cores": int(threads), "kind": "oracle",
            "extrapolated": len(sub) < total,
            "s_per_frame": round(wl.H * wl.W / rate, 2),
            "sample": (f"{len(sub)} rays drawn uniformly (seed 1234) from the {wl.n_poses} x {wl.H} x "
                       f"{wl.W} workload, {wl.precision}-rounding oracle, {dt:.1f} s; the frame time is "
                       f"extrapolated from it" if len(sub) < total else
                       f"all {total} rays of the {wl.n_poses} x {wl.H} x {wl.W} workload, "
                       f"{wl.precision}-rounding oracle, {dt:.1f} s") + f"; os.cpu_count()={os.cpu_count()}"}


def default_cpu_sample(wl):
    """Rays of the oracle's timed sample: 262,144 for the 400 x 400 frames,
    a 65,536-ray subset for the larger workloads (about 7-25 s each)."""
    return 262144 if wl.H * wl.W <= 400 * 400 else 65536


def mfma_loop_ceiling(r, precision, stream, workgroups=2048):
    """TFLOP/s of the library's register-fed MFMA loop in the workload's
    precision (8 waves per SIMD, four independent chains each, random
    operands), timed with events on the render stream after one warm-up."""
    import torch
    iters = {"bf16": 4096, "fp8": 2048, "fp32": 1024}[precision]
    r.mfma_peak(workgroups, iters)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    flop = 0.0
    for _ in range(5):
        flop += r.mfma_peak(workgroups, iters)[1]
    e1.record(stream)
    torch.cuda.synchronize()
    tflops = flop / (e0.elapsed_time(e1) * 1e-3) / 1e12
    log(f"MFMA loop ceiling ({precision}): {tflops:.1f} TFLOP/s")
    return tflops


def bench_targets(args, tw):
    """Training targets (Sec. 5.1, Eq. 6-8) of the seeded depth maps: one
    step is one donerf_targets call over all P maps.  HBM-bound: each pixel
    reads its 4-byte depth once (the window re-reads hit L2) and writes
    4 B bytes of targets."""
    import torch

    from paper_2103_03231_amd import binding as b
    from paper_2103_03231_amd import inputs

    torch.cuda.set_device(0)
    stream = torch.cuda.current_stream()
    r = b.Renderer(b.Config(n_bins=tw.n_bins), inputs.make_weights(tw.n_bins, 0))
    depth_h = inputs.make_depth_maps(tw.P, tw.H, tw.W, tw.seed)
    depth = torch.from_numpy(depth_h).cuda()
    out = torch.empty((tw.P, tw.H, tw.W, tw.n_bins), dtype=torch.float32, device="cuda")
    call = lambda: b.donerf_targets(r.h, depth.data_ptr(), tw.P, tw.H, tw.W, tw.K, tw.Z, out.data_ptr())
    for _ in range(args.warmup):
        call()
    torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    t0 = time.perf_counter()
    for e0, e1 in ev:
        e0.record(stream)
        call()
        e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    kern_ms = float(np.mean([e0.elapsed_time(e1) for e0, e1 in ev]))
    ms_step = wall * 1e3 / args.steps
    bytes_launch = tw.pixels * (4 + 4 * tw.n_bins)
    achieved = bytes_launch / (kern_ms * 1e-3) / 1e9
    line = {
        "metric": "Mpixels/s of depth-oracle training targets (Eq. 6-8)",
        "value": round(tw.pixels / (ms_step * 1e-3) / 1e6, 3), "unit": "Mpixels/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": "synthetic: seeded z-buffered depth maps (tilted discs and rectangles over an empty background)",
        "config": {"workload": tw.name, "maps": tw.P, "H": tw.H, "W": tw.W, "classes": tw.n_bins, "K": tw.K,
                   "Z": tw.Z, "algorithmic_bytes_per_pixel": 4 + 4 * tw.n_bins},
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBS, 4),
                     "traffic": (round(sum(args.traffic_kib) * 1024) if args.traffic_kib else measured_traffic(tw.name)),
                     "kernel": "targets_kernel", "kernel_ms": round(kern_ms, 4)},
    }
    if not args.no_cpu:
        from oracle import targets_oracle as T
        t0 = time.perf_counter()
        for p in range(tw.P):
            T.training_targets(depth_h[p], 0.1, 10.0, tw.n_bins, tw.K, tw.Z)
        dt = time.perf_counter() - t0
        line["cpu_baseline"] = {"value": tw.pixels / dt / 1e6, "unit": "Mpixels/s", "cores": 1, "kind": "oracle",
                                "sample": f"all {tw.P} maps, fp64 NumPy (single-threaded element-wise), {dt:.1f} s"}
    r.close()
    print(json.dumps(line), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="frame400_n4_bf16")
    ap.add_argument("--cpu-sample", type=int, default=None,
                    help="rays of the oracle's timed sample (default: 262,144 for 400 x 400 frames, "
                         "65,536 for larger workloads)")
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--no-mfma-loop", action="store_true",
                    help="skip the register-fed MFMA loop that measures the matrix cores' ceiling")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run a plain device copy of MIB MiB (3 times), to calibrate the "
                         "FETCH_SIZE / WRITE_SIZE counters against known bytes")
    ap.add_argument("--traffic-kib", type=float, nargs=2, default=None, metavar=("FETCH", "WRITE"),
                    help="HBM KiB per render dispatch from the calibrated FETCH_SIZE and WRITE_SIZE "
                         "counters of the current kernel, reported as roofline.traffic")
    args = ap.parse_args()
    if args.copy_calibration:
        import torch
        n = args.copy_calibration * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes_read": n * 4, "bytes_written": n * 4, "repeats": 3}))
        return
    if args.gpus != 1:
        print(json.dumps({"error": "the library runs on one GPU only: the rays of a frame are "
                                   "independent, so several GPUs would each render a share of the "
                                   "image; only --gpus 1 is measured"}))
        sys.exit(2)

    import torch

    from paper_2103_03231_amd import binding as b
    from paper_2103_03231_amd import inputs

    if args.workload in inputs.TARGET_WORKLOADS:
        return bench_targets(args, inputs.TARGET_WORKLOADS[args.workload])
    wl = inputs.WORKLOADS[args.workload]
    weights = inputs.make_weights(wl.n_bins, 0, wl.depth_input)
    poses = wl.poses()
    P = len(poses)
    prec = {"bf16": b.BF16, "fp32": b.FP32, "fp8": b.FP8}[wl.precision]
    sel = {"topn": b.SELECT_TOPN, "topn_softmax": b.SELECT_TOPN_SOFTMAX, "cdf": b.SELECT_CDF}[wl.select]
    torch.cuda.set_device(0)
    stream = torch.cuda.current_stream()
    din = {"encoded": b.DEPTH_ENCODED, "positions": b.DEPTH_POSITIONS}[wl.depth_input]
    r = b.Renderer(b.Config(n_bins=wl.n_bins, n_max=wl.N, precision=prec, fov_x_deg=wl.fov_deg,
                            select=sel, depth_input=din), weights)
    out = r.alloc(P, wl.H, wl.W, wl.N, depth=wl.want_depth)
    log(f"workload {wl.name}: {P} x {wl.H} x {wl.W} rays, N={wl.N}, B={wl.n_bins}, {wl.precision}")

    for _ in range(args.warmup):
        r.render_into(poses, wl.H, wl.W, wl.N, out)
    torch.cuda.synchronize()
    log(f"warmup done ({args.warmup} steps)")

    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for e0, e1 in ev:
        e0.record(stream)
        r.render_into(poses, wl.H, wl.W, wl.N, out)
        e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    kern_ms = [e0.elapsed_time(e1) for e0, e1 in ev]
    avg_kern_ms = float(np.mean(kern_ms))
    log(f"timed {args.steps} steps: wall {wall * 1e3:.2f} ms, kernel avg {avg_kern_ms:.4f} ms")

    loop = mfma_loop_ceiling(r, wl.precision, stream) if not args.no_mfma_loop else None

    rays = wl.rays
    ms_step = wall * 1e3 / args.steps
    value = rays / (ms_step * 1e-3) / 1e6
    d_in = depth_in_folded(wl.depth_input)
    sweeps = 2 if wl.select == "cdf" and wl.n_bins > 128 else 1
    flop_launch = algorithmic_flop_per_ray(wl.N, wl.n_bins, d_in) * rays
    achieved = flop_launch / (avg_kern_ms * 1e-3) / 1e12
    peak = (mixed_peak(wl.N, wl.n_bins, d_in) if wl.precision == "fp8" else MFMA_PEAK_TFLOPS[wl.precision])
    paper_mrays = 400 * 400 / 22e-3 / 1e6   # 22 ms per 400x400 frame, N = 4
    kib = args.traffic_kib
    if kib is not None:
        traffic = round((kib[0] + kib[1]) * 1024)
    else:
        traffic = measured_traffic(wl.name)
    line = {
        "metric": "Mrays/s + ms/frame at 400x400 N=4 (8x256 MLPs); MFMA util % of peak",
        "value": round(value, 3),
        "unit": "Mrays/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "ms_per_frame": round(ms_step / P, 4),
        **({"ms_per_stereo_pair": round(ms_step / (P // 2), 4),
            "stereo_pairs_per_s": round((P // 2) / (ms_step * 1e-3), 3)} if wl.stereo else {}),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": round(value / paper_mrays, 2) if wl.name == "frame400_n4_bf16" else None,
        "dtype": wl.precision,
        "data": "synthetic: seeded cameras on a sphere of radius 1.5 looking at the origin, "
                "He-uniform random-init weights (SplitMix64 seed 0)",
        "config": {"workload": wl.name, "poses": P, "H": wl.H, "W": wl.W, "samples_per_ray": wl.N,
                   "depth_classes": wl.n_bins, "placement": wl.select, "depth_input": wl.depth_input,
                   "rays_per_step": rays,
                   "algorithmic_mflop_per_ray": round(algorithmic_flop_per_ray(wl.N, wl.n_bins, d_in) / 1e6, 4),
                   "padded_mflop_per_ray": round(padded_flop_per_ray(wl.N, wl.n_bins, d_in, sweeps) / 1e6, 4)},
        "roofline": {"bound": "mfma", "achieved": round(achieved, 2), "peak": peak, "unit": "TFLOP/s",
                     "frac": round(achieved / peak, 4),
                     # the same launch counted by the tile work the MFMAs execute (padding included)
                     "padded_frac": round(padded_flop_per_ray(wl.N, wl.n_bins, d_in, sweeps) * rays
                                          / (avg_kern_ms * 1e-3) / 1e12 / peak, 4),
                     **({"peak_note": "fp8 hidden layers at 5000, bf16 first layers and heads at 2500, "
                                      "combined by their share of the work"} if wl.precision == "fp8" else {}),
                     "traffic": traffic,
                     "kernel": f"render_kernel<{wl.precision}>", "kernel_ms": round(avg_kern_ms, 4),
                     "kernel_ms_median": round(float(np.median(kern_ms)), 4)},
    }
    if loop is not None:
        # the measured ceiling: a register-fed MFMA loop on random operands
        line["roofline"]["mfma_loop"] = {"achieved": round(loop, 2), "frac_of_peak":
                                         round(loop / MFMA_PEAK_TFLOPS[wl.precision], 4)}
        if wl.precision != "fp8":   # the fp8 network mixes fp8 and bf16 layers
            line["roofline"]["frac_of_mfma_loop"] = round(achieved / loop, 4)
    if not args.no_cpu:
        line["cpu_baseline"] = cpu_baseline(wl, weights, poses, args.cpu_sample or default_cpu_sample(wl))
    r.close()
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
