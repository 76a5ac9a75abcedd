#!/usr/bin/env python3
"""Sustained decode throughput of the chunked rANS weight decoder on one MI355X.

Workload: Llama-3-70B-shaped decoder layers in bf16 (q/o 8192x8192, k/v
1024x8192, gate/up 28672x8192, down 8192x28672; Normal(0, 0.015) with 0.1 %
outlier input channels x20), 1.711 GB decoded per layer.  `--layers` distinct
layer seeds are drawn on the GPU, encoded on the host with libwc's threaded
encoder (64 KiB chunks, 64 lanes) and kept resident in HBM; every layer is
decoded once and checked byte-exact against its original before timing.

A step is one wc_decode launch that decodes every tensor of one layer from its
resident blob into a resident output buffer (two output sets are ping-ponged);
step k decodes layer k mod --layers.  Each blob (~1.13 GB) is several times the
256 MB Infinity Cache, so every step streams from HBM.  The JSON line reports
decoded GB/s over the K timed steps, the roofline of the decode kernel
(algorithmic bytes = blob bytes read + decoded bytes written, per launch, over
its mean event-timed duration, against 8 TB/s), the compression ratio next to
the order-0 entropy bound, a device-to-device copy ceiling, and the CPU
oracle's single-thread decode rate on the host cores.
"""

from __future__ import annotations

import argparse
import json
import os
import platform
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "decompressed GB/s on one MI355X (% of HBM roofline); ratio vs Shannon bound"
HBM_PEAK_GBPS = 8000.0

# HBM bytes per launch of the 70B-layer decode from rocprofv3 --pmc FETCH_SIZE and
# WRITE_SIZE runs, each scaled by the same counter on a 470 MB device copy (FETCH_SIZE
# reads half the copied bytes: factor 2.0; WRITE_SIZE is exact).  Valid only for
# the kernel source they were taken on (sha256 prefix); otherwise reported as null.
COUNTED_TRAFFIC = {"kernel_sha256": "9781f38eca2731f7", "fetch_bytes": 1142167328,
                   "write_bytes": 1711276848, "chunk_bytes": 65536, "lanes": 64}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or "unknown"


def oracle_baseline(blob, host_tensors):
    """Single-thread oracle decode of one whole layer blob on one host core."""
    import numpy as np

    import oracle
    raw = blob.array()
    info = oracle.tensor_info(raw)
    outs = [np.empty(i["out_bytes"], np.uint8) for i in info]
    old = os.sched_getaffinity(0)
    core = min(old)
    os.sched_setaffinity(0, {core})
    try:
        t0 = time.perf_counter()
        for t, i in enumerate(info):
            oracle.decode_chunks(raw, t, 0, i["n_chunks"], out=outs[t])
        dt = time.perf_counter() - t0
    finally:
        os.sched_setaffinity(0, old)
    for o, h in zip(outs, host_tensors):
        if not np.array_equal(o, h):
            raise RuntimeError("oracle baseline decoded a different layer")
    n_out = sum(i["out_bytes"] for i in info)
    return {"value": round(n_out / dt / 1e9, 4), "unit": "GB/s", "cores": 1, "kind": "oracle",
            "sample": f"layer 0 of the 70B bf16 workload: all {sum(i['n_chunks'] for i in info)} "
                      f"chunks, {n_out} decoded bytes, single thread pinned to core {core}",
            "seconds": round(dt, 3), "cpu": cpu_model(), "host_cpus": os.cpu_count()}


def counted_traffic(chunk_bytes: int, lanes: int):
    import hashlib
    src = os.path.join(ROOT, "paper_2606_15789_amd", "csrc", "wc_decode.hip")
    with open(src, "rb") as fh:
        sha = hashlib.sha256(fh.read()).hexdigest()[:16]
    c = COUNTED_TRAFFIC
    if sha != c["kernel_sha256"] or chunk_bytes != c["chunk_bytes"] or lanes != c["lanes"]:
        return None
    return c["fetch_bytes"] + c["write_bytes"]


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=80)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--layers", type=int, default=8, help="distinct layer seeds resident in HBM")
    ap.add_argument("--chunk-bytes", type=int, default=65536)
    ap.add_argument("--lanes", type=int, default=64)
    ap.add_argument("--threads", type=int, default=int(os.environ.get("OMP_NUM_THREADS", "16")))
    ap.add_argument("--no-cpu-baseline", action="store_true")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU only: the decoder has no multi-GPU path (chunks are "
              "independent and shard with no exchange); run it with --gpus 1.", file=sys.stderr)
        return 2

    import numpy as np
    import torch

    from paper_2606_15789_amd import synth, wc

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 1
    dev = torch.device("cuda:0")
    wc.lib()
    NL = max(1, args.layers)

    # --- setup: draw, encode, upload, verify ---------------------------------
    blobs, dblobs = [], []
    layer_out = None
    sets = None
    err = torch.zeros(1, dtype=torch.int32, device=dev)
    keep_orig = {}
    last_layers = {(args.warmup + args.steps - 1) % NL, (args.warmup + args.steps - 2) % NL}
    comp = None
    cpu = None
    t_setup = time.perf_counter()
    for layer in range(NL):
        t0 = time.perf_counter()
        tens = synth.config_torch_device(5, layer, device="cuda")
        host = [t.cpu().numpy() for _, t, _ in tens]
        blob = wc.encode([("bf16", h) for h in host], chunk_bytes=args.chunk_bytes,
                         lanes=args.lanes, threads=args.threads)
        dblob = wc.to_device(blob, dev)
        if sets is None:
            layer_out = blob.out_bytes
            sets = [[torch.empty(n, dtype=torch.uint8, device=dev) for n in layer_out]
                    for _ in range(2)]
        wc.decode_torch(blob, dblob, outs=sets[0], err=err)
        torch.cuda.synchronize()
        if int(err.item()) != 0:
            raise RuntimeError(f"layer {layer}: device errors {wc.describe_errors(int(err.item()))}")
        for (_, orig, _), out in zip(tens, sets[0]):
            if not torch.equal(orig, out):
                raise RuntimeError(f"layer {layer}: decoded bytes differ from the original")
        if layer in last_layers:
            keep_orig[layer] = [o for _, o, _ in tens]
        if layer == 0:
            stats = [wc.analyze("bf16", h) for h in host]
            bound = sum(st["bound_bytes"] for st in stats)
            raw8 = sum(st["bound_bytes_raw8"] for st in stats)
            out_b = sum(blob.out_bytes)
            comp = {"ratio": round(out_b / blob.size, 5),
                    "bound_ratio": round(out_b / bound, 5),
                    "payload_over_bound_pct": round(100 * (blob.payload_bytes() / bound - 1), 4),
                    "total_over_bound_pct": round(100 * (blob.size / bound - 1), 4),
                    "over_raw8_bound_pct": round(100 * (blob.payload_bytes() / raw8 - 1), 4),
                    "metadata_bytes": blob.breakdown["meta_bytes"]
                    + blob.breakdown["record_hdr_bytes"] + blob.breakdown["pad_bytes"],
                    "breakdown": blob.breakdown}
            if not args.no_cpu_baseline:
                log("cpu baseline: oracle decode of layer 0 on one core ...")
                cpu = oracle_baseline(blob, host)
                log(f"cpu baseline: {cpu['value']} GB/s in {cpu['seconds']} s")
        del tens, host
        blobs.append(blob)
        dblobs.append(dblob)
        log(f"layer {layer + 1}/{NL}: {blob.size / 1e9:.3f} GB compressed, "
            f"{sum(blob.out_bytes) / 1e9:.3f} GB decoded, verified, "
            f"{time.perf_counter() - t0:.1f} s")
    torch.cuda.empty_cache()
    setup_s = time.perf_counter() - t_setup

    # --- device-to-device copy ceiling ----------------------------------------
    src = sets[0][4]
    dst = sets[1][4]
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    c0, c1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    c0.record()
    for _ in range(10):
        dst.copy_(src)
    c1.record()
    torch.cuda.synchronize()
    copy_gbps = 10 * 2 * src.numel() / (c0.elapsed_time(c1) / 1e3) / 1e9

    # --- timed decode ---------------------------------------------------------
    stream = torch.cuda.current_stream(dev)
    err.zero_()

    def step(k):
        layer = k % NL
        outs = sets[k % 2]
        wc.decode(blobs[layer], dblobs[layer].data_ptr(), [o.data_ptr() for o in outs],
                  stream.cuda_stream, err.data_ptr())

    for k in range(args.warmup):
        step(k)
    torch.cuda.synchronize()
    K = args.steps
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(K)]
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record(stream)
    for k in range(K):
        ev[k][0].record(stream)
        step(args.warmup + k)
        ev[k][1].record(stream)
    end.record(stream)
    torch.cuda.synchronize()
    total_ms = start.elapsed_time(end)
    launch_ms = [a.elapsed_time(b) for a, b in ev]

    if int(err.item()) != 0:
        raise RuntimeError(f"device errors during timing: {wc.describe_errors(int(err.item()))}")
    for j in (1, 2):
        k = args.warmup + K - j
        if k < args.warmup:
            continue
        for o, r in zip(sets[k % 2], keep_orig[k % NL]):
            if not torch.equal(o, r):
                raise RuntimeError("timed decode output differs from the original")

    out_per_step = sum(layer_out)
    in_per_step = float(np.mean([b.size for b in blobs]))
    value = K * out_per_step / (total_ms / 1e3) / 1e9
    mean_launch_s = float(np.mean(launch_ms)) / 1e3
    achieved = (in_per_step + out_per_step) / mean_launch_s / 1e9
    line = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": round(total_ms / K, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u32",
        "data": "synthetic",
        "config": {"workload": "llama3-70b-layer-bf16", "layers_resident": NL,
                   "tensors_per_layer": len(layer_out),
                   "decoded_bytes_per_step": out_per_step,
                   "compressed_bytes_per_step": int(in_per_step),
                   "chunk_bytes": args.chunk_bytes, "lanes": args.lanes,
                   "parallelism": "single-gpu"},
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBPS, 4),
                     "traffic": counted_traffic(args.chunk_bytes, args.lanes),
                     "kernel": "wc_decode_kernel",
                     "mean_launch_us": round(mean_launch_s * 1e6, 2),
                     "algorithmic_bytes_per_launch": int(in_per_step + out_per_step)},
        "hbm_pct": round(100 * achieved / HBM_PEAK_GBPS, 2),
        "d2d_copy_GBps": round(copy_gbps, 1),
        "compression": comp,
        "cpu_baseline": cpu,
        "setup_s": round(setup_s, 1),
    }
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
