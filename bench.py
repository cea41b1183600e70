"""Benchmark of the fragment-based image scan on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload ID] [--no-cpu] [--no-cpu-fragment]
                    [--border valid|reflect|symmetric] [--tile R,C]

A step is one full scan (every layer, the head and the reassembly) of the
workload's synthetic image batch, already resident in device memory.  Prints
one JSON line:
  value        output pixels per second (windows classified per second)
  roofline     the launch that takes the most time, its algorithmic work per
               launch over its mean duration (HIP events around repeated
               back-to-back runs of that launch on the scan's stream), against
               the MI355X peak for its bound
  launches     the same for every launch of the scan
  cpu_baseline the per-patch CPU oracle on a deterministic sample of
               windows (every image's corners, the first and last window of
               every final fragment of every image, 4096 seeded random
               windows), on this host's cores
  cpu_fragment the fragment method on the CPU (float64) on the same host, on
               all cores and on one core: the full image when it has at most
               418 x 418 windows, else a top-left crop of image 0 with about
               that many
Default workload: net N4 (the paper's Table 1 net) on a batch of eight
1024 x 1024 greyscale images (8 x 930 x 930 windows), the largest of the
workloads; --workload 2 is the paper's own size, one 512 x 512 slice.
--border reflect / symmetric scans with mirrored edges instead (Section 3.2's
setup: one output per pixel); the per-launch figures then come from the scan
of the extended image.  --tile R,C scans in output tiles (fs_scan_tiled: a
workspace bounded by the tile); the per-launch figures stay those of the
untiled scan.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK = {  # MI355X published dense peaks
    "hbm_gbs": 8000.0,
    "f32_tflops": 157.3,
    "bf16_tflops": 2516.6,
}


def measured_traffic(launch_name, layer, workload):
    """HBM bytes of one launch (the scan's launch of that name and first
    layer) from the committed rocprofv3 counter summary
    (profiles/traffic.json), if it was taken on the current kernel sources;
    else None."""
    from paper_1302_1700_amd.profsum import source_digest
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        entries = json.load(f)
    for e in entries:
        if e.get("launch") == launch_name and e.get("layer") == layer and e.get("workload") == workload \
                and e.get("source_digest") == source_digest():
            return e.get("bytes_per_launch")
    return None


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def oracle_windows(w, n_random=4096, seed=1234):
    """The deterministic window sample of the per-patch baseline: every
    image's corners, the first and the last window of every final fragment
    of every image (from the oracle's corner tracking), and n_random seeded
    random windows; (b, Y, X) rows."""
    import numpy as np
    from oracle import index as ix
    ny, nx = w.out_h, w.out_w
    f = ix.reassembly_index(w.layers, w.height, w.width)[..., 0].ravel()
    _, first = np.unique(f, return_index=True)
    _, last_rev = np.unique(f[::-1], return_index=True)
    flat = np.concatenate([first, f.size - 1 - last_rev])
    rng = np.random.default_rng(seed)
    rows = [np.array([(b, Y, X) for b in range(w.batch) for Y in (0, ny - 1) for X in (0, nx - 1)])]
    for b in range(w.batch):
        rows.append(np.stack([np.full(flat.size, b), flat // nx, flat % nx], 1))
    rows.append(np.stack([rng.integers(0, w.batch, n_random), rng.integers(0, ny, n_random),
                          rng.integers(0, nx, n_random)], 1))
    return np.unique(np.concatenate(rows), axis=0).astype(np.int32)


def cpu_baseline(w, params, img):
    """Per-patch oracle on the deterministic window sample (oracle_windows)."""
    import oracle
    pts = oracle_windows(w)
    n = len(pts)
    t0 = time.perf_counter()
    oracle.patch_forward(w.layers, params, img, w.patch, pts)
    dt = time.perf_counter() - t0
    cores = min(int(os.environ.get("OMP_NUM_THREADS", 0)) or 1 << 30, len(os.sched_getaffinity(0)))
    total = w.batch * w.out_h * w.out_w
    return {
        "value": n / dt,
        "unit": "output px/s",
        "cores": cores,
        "kind": "oracle",
        "cpu_model": cpu_model(),
        "seconds": dt,
        "sample": "%d windows of the same images: corners, the first and last window of every final "
                  "fragment of every image, 4096 seeded random; per-patch float64 forward (C, OpenMP); "
                  "the full map extrapolates to %.0f s" % (n, total / (n / dt)),
    }


def cpu_fragment_baseline(w, params, img, max_windows=418 * 418, one_core=True):
    """The fragment method on the CPU (float64, numpy/BLAS): the full image
    when it has at most max_windows windows, else a top-left crop of image 0
    with about that many; on all cores, then (one_core) the same on one core
    (BLAS limited to one thread)."""
    import oracle
    ny, nx = w.out_h, w.out_w
    sample = "full image"
    if w.batch * ny * nx > max_windows:
        side = int(max_windows ** 0.5)
        ny, nx = min(ny, side), min(nx, side)
        img = img[:1, :ny + w.patch - 1, :nx + w.patch - 1]
        sample = "top-left crop %dx%d of image 0 (%d windows)" % (img.shape[1], img.shape[2], ny * nx)
    n = ny * nx if sample != "full image" else w.batch * ny * nx
    t0 = time.perf_counter()
    oracle.frag_cpu.frag_scan(w.layers, params, img, w.patch)
    dt = time.perf_counter() - t0
    from threadpoolctl import threadpool_info
    blas = [p.get("num_threads", 1) for p in threadpool_info() if p.get("user_api") == "blas"]
    cores = min(max(blas) if blas else 1, len(os.sched_getaffinity(0)))
    res = {"value": n / dt, "unit": "output px/s", "seconds": dt,
           "cores": cores, "kind": "cpu fragment method (float64)",
           "cpu_model": cpu_model(), "sample": sample}
    if one_core:
        from threadpoolctl import threadpool_limits
        with threadpool_limits(limits=1):
            t0 = time.perf_counter()
            oracle.frag_cpu.frag_scan(w.layers, params, img, w.patch)
            dt1 = time.perf_counter() - t0
        res["one_core"] = {"value": n / dt1, "unit": "output px/s", "seconds": dt1, "cores": 1,
                           "sample": sample}
    return res


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=100)
    ap.add_argument("--workload", type=int, default=4)
    ap.add_argument("--profile-reps", type=int, default=10)
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU baseline legs")
    ap.add_argument("--no-cpu-fragment", action="store_true",
                    help="skip the CPU fragment method (timed by default beside the oracle sample)")
    ap.add_argument("--cpu-fragment", action="store_true", help=argparse.SUPPRESS)  # the default
    ap.add_argument("--tile", default=None,
                    help="R,C: scan in output tiles of at most R x C windows (fs_scan_tiled; valid border)")
    ap.add_argument("--border", default="valid", choices=["valid", "reflect", "symmetric"],
                    help="mirrored image edges (one output per pixel)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py: this build runs on exactly one GPU; --gpus %d is not supported" % args.gpus,
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    from paper_1302_1700_amd import fragscan
    from paper_1302_1700_amd import workloads as wl

    w = wl.WORKLOADS[args.workload]
    params, img = wl.workload_inputs(args.workload)
    torch.cuda.set_device(0)
    net = fragscan.Net(w.layers, params, w.channels, 0, w.dtype)
    x = torch.from_numpy(img).cuda()
    border = args.border
    oh, ow = (w.out_h, w.out_w) if border == "valid" else (w.height, w.width)
    out = torch.empty((w.batch, oh, ow, w.n_classes), dtype=torch.float32, device="cuda")
    tile = tuple(int(v) for v in args.tile.split(",")) if args.tile else None
    if tile and border != "valid":
        print("bench.py: --tile scans valid windows only", file=sys.stderr)
        sys.exit(2)
    ws = net.workspace(w.batch, w.height, w.width, x.device, border, tile=tile)

    def step():
        if tile:
            net.scan_tiled(x, tile, out=out, workspace=ws)
        else:
            net.scan(x, out=out, workspace=ws, border=border)
    plan = net.plan(w.batch, w.height, w.width, border)
    # the launches of the (extended) image's scan
    eh, ew = (w.height, w.width) if border == "valid" else (w.height + w.patch - 1, w.width + w.patch - 1)
    launches = net.launches(w.batch, eh, ew)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    t0.record(stream)
    h0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    host_ms = (time.perf_counter() - h0) * 1e3 / args.steps  # enqueue time per scan on the host
    t1.record(stream)
    torch.cuda.synchronize()
    ms = t0.elapsed_time(t1) / args.steps
    pixels = w.batch * oh * ow

    # per-launch mean durations: HIP events around --profile-reps back-to-back
    # runs of each launch on the scan's stream (mirrored borders: the same
    # launches on an image of the extended size; timing does not depend on
    # the pixel values)
    if border == "valid":
        per = net.profile(x, reps=args.profile_reps, out=out)
    else:
        xe = torch.zeros((w.batch, eh, ew, w.channels), dtype=torch.float32, device="cuda")
        xe[:, :w.height, :w.width] = x
        per = net.profile(xe, reps=args.profile_reps)
    peak_mm = PEAK["bf16_tflops"] if w.dtype == "bf16" else PEAK["f32_tflops"]
    rows = []
    for L, t in zip(launches, per):
        r = {"name": L["name"], "layer": L["layer"], "ms": t, "flops": L["flops"], "bytes": L["bytes"],
             "tflops": L["flops"] / (t * 1e-3) / 1e12 if t > 0 else 0.0,
             "gbs": L["bytes"] / (t * 1e-3) / 1e9 if t > 0 else 0.0}
        ai = L["flops"] / L["bytes"] if L["bytes"] else 0.0
        ridge = peak_mm * 1e12 / (PEAK["hbm_gbs"] * 1e9)
        r["bound"] = "mfma" if ai >= ridge else "hbm"
        r["frac"] = r["tflops"] / peak_mm if r["bound"] == "mfma" else r["gbs"] / PEAK["hbm_gbs"]
        rows.append(r)
    dom = max(rows, key=lambda r: r["ms"])
    conv_flops = sum(r["flops"] for r in rows)
    conv_ms = sum(r["ms"] for r in rows if r["flops"] > 0)
    traffic = measured_traffic(dom["name"], dom["layer"], w.name) if border == "valid" else None
    if dom["bound"] == "mfma":
        roof = {"bound": "mfma", "achieved": dom["tflops"], "peak": peak_mm, "unit": "TFLOP/s",
                "frac": dom["tflops"] / peak_mm}
    else:
        roof = {"bound": "hbm", "achieved": dom["gbs"], "peak": PEAK["hbm_gbs"], "unit": "GB/s",
                "frac": dom["gbs"] / PEAK["hbm_gbs"]}
    roof["traffic"] = traffic
    roof["kernel"] = dom["name"]
    roof["layer"] = dom["layer"]
    roof["work_per_launch"] = dom["flops"] if dom["bound"] == "mfma" else dom["bytes"]
    roof["mean_launch_ms"] = dom["ms"]

    res = {
        "metric": "output pixels/sec per image scan (1 GPU) + conv TFLOP/s as % MFMA peak",
        "value": pixels / (ms * 1e-3),
        "unit": "output px/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if w.dtype == "bf16" else "f32",
        "data": "synthetic",
        "config": {"workload": w.name, "image": [w.batch, w.height, w.width, w.channels],
                   "patch": w.patch, "outputs": [w.batch, oh, ow], "fragments": net.info["n_fragments"],
                   "border": border, "tile": list(tile) if tile else None,
                   "workspace_bytes": ws.numel()},
        "host_enqueue_ms_per_step": host_ms,
        "tflops": plan["flops"] / (ms * 1e-3) / 1e12,
        "pct_mfma_peak": 100.0 * plan["flops"] / (ms * 1e-3) / 1e12 / peak_mm,
        "conv_tflops_in_conv_kernels": conv_flops / (conv_ms * 1e-3) / 1e12 if conv_ms else 0.0,
        "roofline": roof,
        "launches": rows,
    }
    net.close()
    if not args.no_cpu:
        res["cpu_baseline"] = cpu_baseline(w, params, img)
        if not args.no_cpu_fragment and border == "valid" and not tile:
            res["cpu_fragment"] = cpu_fragment_baseline(w, params, img)
    print(json.dumps(res))


if __name__ == "__main__":
    main()
