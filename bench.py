"""Benchmark: feature-extraction images/sec to the split layer on one MI355X.

Default workload: ResNet-50 (Bottleneck [3, 4, 6, 3]), inference batch-norm
folded, bf16 weights and activations with fp32 accumulation, batch 256 of
synthetic 3x224x224 images, split after layer4 (2048x7x7, layer 18).  One step
is one ``hapi_extract`` call over the whole batch: every layer from the input
to the split, plus writing the split activations in NCHW; by default the
library runs it as two 128-image partitions in flight on two streams.
Weights are packed once beforehand (model reuse); images and weights are
resident in HBM.

Prints ONE JSON line with the throughput, the share of the step's MFMA
capacity the convolutions used, a roofline entry for the dominant kernel
family (HIP events recorded by each launch on the stream it runs on) and the
CPU oracle timed on a bounded sample as a baseline.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

PEAK = {"bf16": 2500.0, "f32": 157.3}  # dense MFMA TFLOP/s (MI355X)
# Sources of the convolution kernel family whose counters the traffic profile holds.
CONV_SOURCES = ("conv.hip", "conv3x3.hip", "stem.hip", "bottleneck.hip")
HBM_PEAK = 8000.0                      # GB/s


def _cores():
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    omp = os.environ.get("OMP_NUM_THREADS")
    return min(n, int(omp)) if omp and omp.isdigit() else n


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def _sclk_now():
    """Highest current shader clock (MHz) over the GPUs' sysfs DPM tables
    (the line marked '*'), or None when unreadable."""
    import glob
    import re
    best = None
    for path in glob.glob("/sys/class/drm/card*/device/pp_dpm_sclk"):
        try:
            for line in open(path):
                if "*" in line:
                    m = re.search(r"(\d+)\s*[Mm][Hh]z", line)
                    if m:
                        best = max(best or 0, int(m.group(1)))
        except OSError:
            pass
    return best


def sustained_sclk(step, seconds=1.5):
    """Median shader clock sampled every 20 ms while the workload runs back to
    back for about `seconds` (outside the timed region)."""
    import threading
    import torch
    samples, stop = [], threading.Event()

    def sampler():
        while not stop.is_set():
            v = _sclk_now()
            if v:
                samples.append(v)
            time.sleep(0.02)

    torch.cuda.synchronize()
    th = threading.Thread(target=sampler, daemon=True)
    th.start()
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < seconds:
        for _ in range(20):
            step()
        torch.cuda.synchronize()
    stop.set()
    th.join()
    if not samples:
        return None, 0
    samples.sort()
    return samples[len(samples) // 2], len(samples)


def measured_traffic(workload):
    """HBM bytes per convolution launch from the committed rocprofv3 counter
    summary, or None when a convolution source changed since it was taken."""
    import hashlib
    root = os.path.dirname(os.path.abspath(__file__))
    path = os.path.join(root, "profiles", "conv_bf16_resnet50_b256_hbm_traffic.md")
    if workload != "resnet50_bf16_b256" or not os.path.exists(path):
        return None
    kv = dict(line.strip().split("=", 1) for line in open(path) if "=" in line and " " not in line.strip())
    h = hashlib.sha256()
    try:
        for name in CONV_SOURCES:
            h.update(open(os.path.join(root, "paper_2210_08650_amd", "csrc", name), "rb").read())
    except OSError:  # sources not shipped: the counters cannot be matched to the kernels
        return None
    if h.hexdigest() != kv.get("conv_source_sha256"):
        return None
    return float(kv["conv_traffic_bytes_per_launch"])


def cpu_baseline(cfg, budget_s=15.0):
    """The oracle on a bounded sample of the same workload (images/sec)."""
    import synth
    from oracle import layers as OL
    from oracle import models as OM
    threads = _cores()
    OL.set_threads(threads)
    om = OM.build(cfg["model"])
    ps = synth.params(cfg["seed"], om.manifest())
    imgs = synth.images(cfg["seed"], min(cfg["batch"], 64))
    if cfg["dtype_name"] == "bf16":  # the oracle sees the bf16 values the GPU consumes
        import torch
        imgs = torch.from_numpy(imgs).to(torch.bfloat16).float().numpy()
    t0 = time.perf_counter()
    om.forward(ps, imgs[:1], cfg["split"])
    t1 = time.perf_counter() - t0
    n = int(max(1, min(len(imgs) - 1, budget_s / max(t1, 1e-3))))
    t0 = time.perf_counter()
    om.forward(ps, imgs[1:1 + n], cfg["split"])
    dt = time.perf_counter() - t0
    return {"value": round(n / dt, 4), "unit": "images/s", "cores": threads, "cpu": cpu_model(), "kind": "oracle",
            "sample": f"{n} images of the same workload (images 1..{n}), float64 oracle, "
                      f"{dt:.1f} s"}


def concurrent_requests(args):
    """The storage server's request pattern: each step serves ``requests``
    requests of ``request_images`` images (one training iteration), split into
    storage-side partitions of ``chunk`` images (default 16), with
    ``concurrency`` requests in flight at once, each on its own stream and
    workspace, issued by its own host thread."""
    import threading
    import torch
    import paper_2210_08650_amd as H
    from paper_2210_08650_amd import models as PM
    import synth

    cfg = dict(PM.WORKLOADS[args.workload])
    S, R, Q = args.concurrency, args.requests, args.request_images
    chunk = args.chunk or 16
    layers = PM.FACTORIES[cfg["model"]]()
    tdt = torch.bfloat16 if cfg["dtype"] == H.HAPI_BF16 else torch.float32
    split = cfg["split"]
    streams = [torch.cuda.Stream() for _ in range(S)]
    descs, spaces = [], []
    for t in range(S):
        d = H.Desc(layers, cfg["dtype"], stream=streams[t], chunk=chunk)
        need = H.hapi_workspace_bytes(d, Q, split)
        spaces.append(torch.empty(max(need, 256), dtype=torch.uint8, device="cuda"))
        descs.append(d.set(workspace=spaces[t], workspace_bytes=need))
    raw = torch.from_numpy(synth.flatten(synth.params(cfg["seed"], PM.raw_manifest(layers)))).cuda()
    packed = torch.empty(H.hapi_packed_weight_bytes(descs[0]), dtype=torch.uint8, device="cuda")
    H.hapi_pack_weights(H.Desc(layers, cfg["dtype"]), raw, packed)
    images = torch.from_numpy(synth.images(cfg["seed"], R * Q)).to(tdt).cuda()
    out = torch.empty((R, Q) + H.hapi_layer_shape(descs[0], split), dtype=tdt, device="cuda")
    torch.cuda.synchronize()
    del raw

    def worker(t):
        for i in range(t, R, S):
            H.hapi_extract(descs[t], packed, images[i * Q:(i + 1) * Q], Q, split, out[i])

    def step():
        th = [threading.Thread(target=worker, args=(t,)) for t in range(S)]
        for x in th:
            x.start()
        for x in th:
            x.join()

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    print(json.dumps({
        "metric": f"feature-extraction images/sec, {R} requests of {Q} images, "
                  f"{S} in flight ({cfg['model']})",
        "value": round(R * Q * args.steps / elapsed, 2), "unit": "images/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(elapsed * 1e3 / args.steps, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16" if cfg["dtype"] == H.HAPI_BF16 else "f32", "data": "synthetic",
        "config": {"workload": args.workload, "requests": R, "request_images": Q,
                   "concurrency": S, "chunk": chunk, "split_layer": split}}), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="resnet50_bf16_b256")
    ap.add_argument("--batch", type=int, default=0, help="override the workload batch")
    ap.add_argument("--chunk", type=int, default=0)
    ap.add_argument("--inflight", type=int, default=0,
                    help="partitions in flight on separate streams (0: the library chooses)")
    ap.add_argument("--direct", action="store_true",
                    help="launch every kernel on every step (no replay of a captured HIP graph)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-sclk", action="store_true",
                    help="skip the sustained run that samples the shader clock (for profiler runs)")
    ap.add_argument("--calib-copy", action="store_true",
                    help="time the library's plain copy (split 0) instead, for counter calibration")
    ap.add_argument("--concurrency", type=int, default=0,
                    help="server mode: --requests requests of --request-images images per step, "
                         "issued by this many host threads on as many streams")
    ap.add_argument("--requests", type=int, default=8)
    ap.add_argument("--request-images", type=int, default=128)
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for {args.gpus}); the extraction shards "
              "by images across GPUs with no communication, see the design notes.", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2210_08650_amd as H
    from paper_2210_08650_amd import models as PM
    import synth

    if args.concurrency:
        return concurrent_requests(args)

    cfg = dict(PM.WORKLOADS[args.workload])
    if args.batch:
        cfg["batch"] = args.batch
    cfg["dtype_name"] = "bf16" if cfg["dtype"] == H.HAPI_BF16 else "f32"
    split = 0 if args.calib_copy else cfg["split"]
    layers = PM.FACTORIES[cfg["model"]]()
    B = cfg["batch"]
    stream = torch.cuda.current_stream()
    desc = H.Desc(layers, cfg["dtype"], stream=stream, chunk=args.chunk, inflight=args.inflight,
                  direct=int(args.direct))
    tdt = torch.bfloat16 if cfg["dtype"] == H.HAPI_BF16 else torch.float32

    raw = torch.from_numpy(synth.flatten(synth.params(cfg["seed"], PM.raw_manifest(layers)))).cuda()
    packed = torch.empty(H.hapi_packed_weight_bytes(desc), dtype=torch.uint8, device="cuda")
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    H.hapi_pack_weights(desc, raw, packed)
    torch.cuda.synchronize()
    load_ms = (time.perf_counter() - t0) * 1e3
    del raw
    images = torch.from_numpy(synth.images(cfg["seed"], B)).to(tdt).cuda()
    out = torch.empty((B,) + H.hapi_layer_shape(desc, split), dtype=tdt, device="cuda")
    ws_bytes = H.hapi_workspace_bytes(desc, B, split)
    ws = torch.empty(max(ws_bytes, 256), dtype=torch.uint8, device="cuda")
    desc.set(workspace=ws, workspace_bytes=ws_bytes)

    def step():
        H.hapi_extract(desc, packed, images, B, split, out)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    ms_per_step = elapsed * 1e3 / args.steps

    # Per-kernel timing: HIP events around every launch, on the library's stream.
    H.hapi_stats_enable(True)
    t1 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    stats_elapsed = time.perf_counter() - t1
    stats = H.hapi_stats_collect()
    H.hapi_stats_enable(False)
    fam = {s["name"]: s for s in stats}
    conv_name = "conv_bf16" if cfg["dtype"] == H.HAPI_BF16 else "conv_f32"
    total_kernel_ms = sum(s["total_ms"] for s in stats)
    if args.calib_copy:
        c = fam["copy"]
        dom, bound, unit = c, "hbm", "GB/s"
        achieved = c["bytes"] / (c["total_ms"] * 1e-3) / 1e9
        peak = HBM_PEAK
    else:
        # Partitions in flight overlap their launches: the family's rate is its
        # flops over the time at least one of its launches was running
        # (equal to the summed durations when nothing overlaps).
        dom = fam[conv_name]
        bound, unit = "mfma", "TFLOP/s"
        achieved = dom["flops"] / (dom["busy_ms"] * 1e-3) / 1e12
        peak = PEAK[cfg["dtype_name"]]
    # share of the whole step's MFMA capacity the convolutions used
    mfma_util = None if args.calib_copy else round(
        100.0 * dom["flops"] / args.steps / (ms_per_step * 1e-3) / 1e12 / peak, 2)

    sclk, sclk_n = (None, 0) if args.calib_copy or args.no_sclk else sustained_sclk(step)

    default = args.workload == "resnet50_bf16_b256" and not args.batch and not args.calib_copy
    result = {
        "metric": ("feature-extraction images/sec to split layer (ResNet-50 bf16 b=256); MFMA util %"
                   if default else f"feature-extraction images/sec to split layer ({args.workload}, "
                                   f"batch {B})"),
        "value": round(B * args.steps / elapsed, 2),
        "unit": "images/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg["dtype_name"],
        "data": "synthetic (seeded N(0,1) images, He-init weights with seeded BN statistics)",
        "config": {"workload": args.workload + ("_copy_calibration" if args.calib_copy else ""),
                   "batch": B, "split_layer": split, "image": "3x224x224",
                   "chunk": args.chunk or "auto",
                   "partitions": H.hapi_chunk_count(desc, B),
                   "inflight": args.inflight or "auto",
                   "launch": "direct" if args.direct else "graph replay"},
        "mfma_util_pct": mfma_util,
        # the same share against the peak at the shader clock measured while
        # the workload ran (datasheet peaks assume 2.4 GHz)
        "sclk_mhz": sclk,
        "sclk_samples": sclk_n,
        "mfma_util_pct_at_sclk": (round(mfma_util * 2400.0 / sclk, 2) if mfma_util is not None and sclk
                                  else None),
        "roofline": {"bound": bound, "achieved": round(achieved, 2), "peak": peak, "unit": unit,
                     "peak_at_sclk": (round(peak * sclk / 2400.0, 1) if bound == "mfma" and sclk else None),
                     "frac": round(achieved / peak, 4),
                     "traffic": None if args.calib_copy or args.batch else measured_traffic(args.workload),
                     "algorithmic_bytes_per_launch": round(dom["bytes"] / dom["launches"]),
                     "algorithmic_flops_per_launch": round(dom["flops"] / dom["launches"]),
                     "kernel": dom["name"], "launches_per_step": dom["launches"] // args.steps,
                     "avg_launch_us": round(dom["total_ms"] * 1e3 / dom["launches"], 2),
                     "busy_us_per_launch": round(dom["busy_ms"] * 1e3 / dom["launches"], 2),
                     "share_of_kernel_time": round(dom["total_ms"] / total_kernel_ms, 4)},
        "kernel_families": {s["name"]: {"ms_per_step": round(s["total_ms"] / args.steps, 4),
                                        "busy_ms_per_step": round(s["busy_ms"] / args.steps, 4),
                                        "launches_per_step": s["launches"] // args.steps}
                            for s in stats},
        "stats_pass_ms_per_step": round(stats_elapsed * 1e3 / args.steps, 4),
        "model_load_ms": round(load_ms, 3),
    }
    if not args.no_cpu_baseline and not args.calib_copy:
        result["cpu_baseline"] = cpu_baseline(cfg)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
