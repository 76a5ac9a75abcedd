#!/usr/bin/env python3
"""Decode throughput of the chunked rANS weight decoder on one MI355X.

Workloads (`--workload`, seeded synthetic tensors with the shapes and
statistics of the paper's models):
  llama3-70b-layer-bf16 (default)  q/o 8192x8192, k/v 1024x8192, gate/up
      28672x8192, down 8192x28672, Normal(0, 0.015) with 0.1 % outlier input
      channels x20; 1.711 GB decoded per layer; `--layers` distinct layer
      seeds are drawn on the GPU and kept resident;
  bf16-matrix-4096        one 4096x4096 bf16 matrix, Normal(0, 0.02);
  llama3-8b-layer-bf16    one Llama-3-8B layer in bf16 (outlier channels);
  llama3-8b-layer-int4    the same shapes as int4 codes (group 128) + fp16
      scales + bf16 norms;
  llama3-8b-layer-int8    the same shapes as per-row int8 (Student-t weights)
      + fp16 scales + bf16 norms;
  llama3-8b-layer-fp8-e4m3  fp8 e4m3 codes with per-row bf16 scales;
  llama3-8b-layer-mxfp4   fp4 e2m1 codes + e8m0 scales per 32 inputs;
  llama3-8b-layer-awq4    4-bit codes + 4-bit zero points + fp16 scales, g128.
Blobs are encoded on the host with libwc's threaded encoder (64 KiB chunks,
64 lanes by default) and kept resident in HBM; every resident blob is decoded
once and checked byte-exact against its original before timing.

A step of the 70B workload decodes every resident layer (80 by default, the
whole model), one wc_decode launch per layer, back to back on one stream into
two ping-ponged output sets: the sustained run.  Each layer blob is ~1.13 GB,
several times the 256 MB Infinity Cache.  A step of the smaller workloads is
one wc_decode launch of one of enough resident copies of the blob and output
set (at least 1 GiB together) that every launch streams from HBM.  A launch
decodes every tensor of its blob.  The JSON line reports decoded GB/s over the
K timed steps; the roofline of the decode kernel (algorithmic bytes = blob
bytes read + decoded bytes written, per launch, over the median of the
event-timed launch durations, against 8 TB/s); the ceiling that a plain
streaming kernel (wc_stream) reaches on the same byte mix, and torch's device
copy; the compression ratio next to the order-0 entropy bound; the CPU
oracle's decode rate on one host core and on all of them; and, with
--two-stream, the same steps with consecutive launches on two streams.
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
MFMA_BF16_PEAK_TFLOPS = 2500.0   # MI355X dense bf16 matrix peak
WORKLOAD_DEFAULT = "llama3-70b-layer-bf16"
# workload name -> seeded recipe number in paper_2606_15789_amd.synth.config
WORKLOADS = {WORKLOAD_DEFAULT: 5, "bf16-matrix-4096": 1, "llama3-8b-layer-bf16": 2,
             "llama3-8b-layer-int4": 3, "llama3-8b-layer-int8": 4,
             "llama3-8b-layer-fp8-e4m3": 6, "llama3-8b-layer-mxfp4": 7,
             "llama3-8b-layer-awq4": 8, "llama3-8b-layer-fp8-e5m2": 9}
ROTATE_BYTES = 1 << 30   # resident bytes the small workloads rotate over

# HBM bytes per launch of a workload's decode (64 KiB chunks, 64 lanes, untiled,
# per-tensor tables) from rocprofv3 --pmc FETCH_SIZE and WRITE_SIZE runs, each scaled
# by the same counter on a 512 MiB device copy (FETCH_SIZE reads half the copied
# bytes: factor 2.0; WRITE_SIZE is exact).  Valid only for the kernel and code they
# were taken on (its fingerprint, the hash of its gfx950 assembly that the build
# writes); otherwise reported as null.
COUNTED_TRAFFIC = {
    "llama3-70b-layer-bf16": {"kernel": "wc_decode_kernel", "kernel_fingerprint": "26a86b454521e29a",
                              "fetch_bytes": 1141265856, "write_bytes": 1738020407},
    "llama3-8b-layer-bf16": {"kernel": "wc_decode_wide_kernel",
                             "kernel_fingerprint": "f89c395c2a6474d3",
                             "fetch_bytes": 291863961, "write_bytes": 443041996},
}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def cpu_model() -> str:
    """The host CPU as /proc/cpuinfo names it, with its family / model /
    stepping numbers (some hosts report only a short vendor name)."""
    info = {}
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if ":" in line:
                    k, v = (x.strip() for x in line.split(":", 1))
                    if k in ("model name", "cpu family", "model", "stepping", "vendor_id") \
                            and k not in info:
                        info[k] = v
                if not line.strip() and info:
                    break
    except OSError:
        pass
    name = info.get("model name") or platform.processor() or "unknown"
    ids = ", ".join(f"{k} {info[k]}" for k in ("vendor_id", "cpu family", "model", "stepping")
                    if k in info)
    return f"{name} ({ids})" if ids else name


def oracle_baseline(blob, host_tensors, workload: str, rep_seconds: float = 3.0):
    """The oracle's decode of one whole blob, timed around the decode calls only.

    One core: the process pinned to one host core, three repetitions, each
    decoding the blob as many times as it takes to pass `rep_seconds` (at
    least once); the median of the three rates.  All cores: the chunks of every
    tensor split into one contiguous range per available core, one thread per
    range (the oracle's C calls release the interpreter lock), three timed
    whole-blob decodes, the median.  Both outputs are checked against the
    original tensors.
    """
    import threading

    import numpy as np

    import oracle
    raw = blob.array()
    info = oracle.tensor_info(raw)
    outs = [np.empty(i["out_bytes"], np.uint8) for i in info]
    n_out = sum(i["out_bytes"] for i in info)
    n_chunks = sum(i["n_chunks"] for i in info)
    old = os.sched_getaffinity(0)
    core = min(old)

    def check():
        for o, h in zip(outs, host_tensors):
            if not np.array_equal(o, np.ascontiguousarray(h).view(np.uint8).reshape(-1)):
                raise RuntimeError("oracle baseline decoded a different blob")

    os.sched_setaffinity(0, {core})
    rates, total, reps_each = [], 0.0, []
    try:
        for _ in range(3):
            reps, dt = 0, 0.0
            while reps == 0 or dt < rep_seconds:
                t0 = time.perf_counter()
                for t, i in enumerate(info):
                    oracle.decode_chunks(raw, t, 0, i["n_chunks"], out=outs[t])
                dt += time.perf_counter() - t0
                reps += 1
            rates.append(reps * n_out / dt / 1e9)
            reps_each.append(reps)
            total += dt
    finally:
        os.sched_setaffinity(0, old)
    check()
    what = "layer 0 of the 70B bf16 workload" if workload == WORKLOAD_DEFAULT else workload
    one = {"value": round(float(np.median(rates)), 4), "unit": "GB/s", "cores": 1,
           "kind": "oracle",
           "sample": f"{what}: all {n_chunks} chunks, {n_out} decoded bytes; three timed "
                     f"repetitions of {reps_each} whole-blob decodes, median rate; single "
                     f"thread pinned to core {core}",
           "runs_GBps": [round(r, 4) for r in rates], "seconds": round(total, 3),
           "cpu": cpu_model(), "host_cpus": os.cpu_count()}

    # all cores: disjoint chunk ranges, one thread each
    cores = sorted(old)
    jobs = [[] for _ in cores]
    for t, i in enumerate(info):
        n = i["n_chunks"]
        for k in range(len(cores)):
            c0, c1 = n * k // len(cores), n * (k + 1) // len(cores)
            if c1 > c0:
                jobs[k].append((t, c0, c1))
    for o in outs:
        o.fill(0)
    errs = []

    def work(k):
        try:
            os.sched_setaffinity(0, {cores[k]})
            for t, c0, c1 in jobs[k]:
                oracle.decode_chunks(raw, t, c0, c1, out=outs[t])
        except Exception as e:  # noqa: BLE001
            errs.append(e)

    walls = []
    for _ in range(3):
        ths = [threading.Thread(target=work, args=(k,)) for k in range(len(cores))]
        t0 = time.perf_counter()
        for th in ths:
            th.start()
        for th in ths:
            th.join()
        walls.append(time.perf_counter() - t0)
    os.sched_setaffinity(0, old)
    if errs:
        raise errs[0]
    check()
    allc = {"value": round(n_out / float(np.median(walls)) / 1e9, 4), "unit": "GB/s",
            "cores": len(cores), "kind": "oracle",
            "sample": f"{what}: the same blob, its chunks split into {len(cores)} contiguous "
                      "ranges per tensor, one thread per range pinned to its own core; three "
                      "timed whole-blob decodes, median",
            "seconds": round(sum(walls), 3)}
    return one, allc


def oracle_gemv_baseline(blob, w0, M: int, layer_weight_bytes: int, min_seconds: float = 10.0):
    """Single-thread oracle of the fused decode-GEMM on one host core, on a
    bounded sample: the oracle decode of the first tensor's tiles and its fp64
    product with up to 2 rows of x, repeated for at least `min_seconds`; the
    per-byte decode time and the per-byte, per-row product time are scaled to
    the whole layer at M rows."""
    import numpy as np

    import oracle
    raw = blob.array()
    info = oracle.tensor_info(raw)[0]
    out = np.empty(info["out_bytes"], np.uint8)
    rows = min(M, 2)
    x = (np.random.default_rng(7).normal(0, 1, (rows, w0.shape[1])).astype(np.float32)
         .view(np.uint32) >> 16).astype(np.uint16)
    old = os.sched_getaffinity(0)
    core = min(old)
    os.sched_setaffinity(0, {core})
    reps, t_dec, t_mul = 0, 0.0, 0.0
    try:
        while reps == 0 or t_dec + t_mul < min_seconds:
            t0 = time.perf_counter()
            oracle.decode_chunks(raw, 0, 0, info["n_chunks"], out=out)
            t1 = time.perf_counter()
            oracle.gemv_bf16(out.view(np.uint16).reshape(w0.shape), x)
            t_mul += time.perf_counter() - t1
            t_dec += t1 - t0
            reps += 1
    finally:
        os.sched_setaffinity(0, old)
    if not np.array_equal(out, np.ascontiguousarray(w0).view(np.uint8).reshape(-1)):
        raise RuntimeError("oracle baseline decoded a different tensor")
    wb = info["out_bytes"]
    step_s = (t_dec / reps / wb + t_mul / reps / rows / wb * M) * layer_weight_bytes
    return {"value": round(layer_weight_bytes / step_s / 1e9, 5), "unit": "GB/s", "cores": 1,
            "kind": "oracle",
            "sample": f"tensor 0 ({w0.shape[0]}x{w0.shape[1]} bf16, {info['n_chunks']} tiles): "
                      f"oracle decode + fp64 product with {rows} x row(s), {reps}x; per-byte "
                      f"decode and per-byte-per-row product times scaled to the layer's "
                      f"{layer_weight_bytes} weight bytes at M = {M}; single thread pinned to "
                      f"core {core}",
            "seconds": round(t_dec + t_mul, 3), "cpu": cpu_model(), "host_cpus": os.cpu_count()}


def rotation_copies(nbytes_per_copy: int) -> int:
    """Resident copies of a step's operands so that consecutive steps never
    find them in the 256 MB Infinity Cache: at least ROTATE_BYTES together,
    and at least two."""
    return max(2, -(-ROTATE_BYTES // max(1, int(nbytes_per_copy))))


def timed_rotating(fn, warmup: int, steps: int, stream) -> float:
    """Mean seconds per step of fn(k), k counting the steps (warm-up first),
    between two events on `stream`."""
    import torch
    for k in range(warmup):
        fn(k)
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record(stream)
    for k in range(steps):
        fn(warmup + k)
    b.record(stream)
    torch.cuda.synchronize()
    return a.elapsed_time(b) / steps / 1e3


def hbm_read_rate(dev, stream) -> float:
    """GB/s of wc_stream reading 1 GiB once (no writes), median of 10."""
    import numpy as np
    import torch

    from paper_2606_15789_amd import wc
    buf = torch.zeros(1 << 30, dtype=torch.uint8, device=dev)
    sink = torch.zeros(16, dtype=torch.uint8, device=dev)
    for _ in range(2):
        wc.stream_bytes(buf.data_ptr(), buf.numel(), sink.data_ptr(), 0, 0, stream.cuda_stream)
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(10)]
    for e0, e1 in ev:
        e0.record(stream)
        wc.stream_bytes(buf.data_ptr(), buf.numel(), sink.data_ptr(), 0, 0, stream.cuda_stream)
        e1.record(stream)
    torch.cuda.synchronize()
    med = float(np.median([e0.elapsed_time(e1) for e0, e1 in ev])) / 1e3
    del buf
    torch.cuda.empty_cache()
    return (1 << 30) / med / 1e9


def kernel_fingerprint(name: str = "wc_decode_kernel"):
    """The fingerprint of a kernel's gfx950 code in the loaded library (written
    next to it by the build), or None."""
    from paper_2606_15789_amd import wc
    path = os.path.splitext(wc.library_path())[0] + ".kernels.json"
    try:
        with open(path) as fh:
            prints = json.load(fh)
    except (OSError, ValueError):
        return None
    return next((v for k, v in prints.items() if name in k), None)


def decode_kernel_for(dtypes, n_chunks: int, lanes: int, tiled: bool) -> str:
    """The kernel wc_decode runs for one launch of these tensors: its 16-wave
    kernel for bf16/fp16 tensors in untiled 64-lane chunks when the chunks
    exceed the general kernel's resident waves (24 a compute unit: the LDS of
    three 8-wave workgroups) but fit the 16-wave kernel's (32 a compute unit),
    the general kernel otherwise.  The library takes the same decision from the
    runtime's occupancy figures."""
    import torch
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    if (all(d in ("bf16", "fp16") for d in dtypes) and lanes == 64 and not tiled
            and 24 * cus < n_chunks <= 32 * cus):
        return "wc_decode_wide_kernel"
    return "wc_decode_kernel"


def gemv_kernel_for(weights: str, n_tiles: int, m: int) -> str:
    """The kernel of a fused-GEMM launch of 16-row tiles (weights: "bf16",
    "int8", "e4m3", "e5m2", or "mxfp4" / "int4" with "-bytes" when the 4-bit
    codes are coded as bytes).  bf16, int8, fp8 and byte-coded 4-bit launches
    take a 16-wave
    kernel when they have up to 16 rows of x (8 for the 4-bit codes) and their
    tiles exceed the 8-wave kernel's resident waves (24 a compute unit) but fit
    the 16-wave kernel's (32 a compute unit).  The library takes the same
    decision from the runtime's occupancy figures."""
    import torch
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    wide_rows = {"bf16": 16, "int8": 16, "e4m3": 16, "e5m2": 16, "mxfp4-bytes": 8,
                 "int4-bytes": 8}
    wide = m <= wide_rows.get(weights, 0) and 24 * cus < n_tiles <= 32 * cus
    general = {"bf16": "wc_gemv_kernel (bf16)", "int8": "wc_gemv_kernel (int8)",
               "e4m3": "wc_gemv_kernel (fp8 e4m3)",
               "e5m2": "wc_gemv_e5m2_kernel", "mxfp4": "wc_gemv_mx_kernel",
               "mxfp4-bytes": "wc_gemv_mxb_kernel", "int4": "wc_gemv_w4n_kernel",
               "int4-bytes": "wc_gemv_w4_kernel"}[weights]
    if not wide:
        return general
    return {"bf16": "wc_gemv_wide_bf16_kernel", "int8": "wc_gemv_wide_kernel (int8)",
            "e4m3": "wc_gemv_wide_kernel (fp8 e4m3)",
            "e5m2": "wc_gemv_wide_e5m2_kernel", "mxfp4-bytes": "wc_gemv_wide_q4_kernel (MXFP4)",
            "int4-bytes": "wc_gemv_wide_q4_kernel (int4)"}[weights]


def counted_traffic(workload: str, chunk_bytes: int, lanes: int, tiled: bool, kernel: str):
    """HBM bytes per launch from the counter runs, if they were taken on this
    workload and layout and on the kernel the launch runs on, as built now."""
    c = COUNTED_TRAFFIC.get(workload)
    if (c is None or tiled or chunk_bytes != 65536 or lanes != 64 or kernel != c["kernel"]
            or kernel_fingerprint(kernel) != c["kernel_fingerprint"]):
        return None
    return c["fetch_bytes"] + c["write_bytes"]


def compression_stats(blob, typed_host):
    """Compressed size against the field-wise order-0 bound of every tensor."""
    from paper_2606_15789_amd import wc
    stats = [wc.analyze(dt, h) for dt, h in typed_host]
    bound = sum(st["bound_bytes"] for st in stats)
    raw8 = sum(st["bound_bytes_raw8"] for st in stats)
    out_b = sum(blob.out_bytes)
    return {"ratio": round(out_b / blob.size, 5),
            "bound_ratio": round(out_b / bound, 5),
            "payload_over_bound_pct": round(100 * (blob.payload_bytes() / bound - 1), 4),
            "total_over_bound_pct": round(100 * (blob.size / bound - 1), 4),
            "over_raw8_bound_pct": round(100 * (blob.payload_bytes() / raw8 - 1), 4),
            "metadata_bytes": blob.breakdown["meta_bytes"]
            + blob.breakdown["record_hdr_bytes"] + blob.breakdown["pad_bytes"],
            "breakdown": blob.breakdown}


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", choices=list(WORKLOADS), default=WORKLOAD_DEFAULT)
    ap.add_argument("--layers", type=int, default=80,
                    help="distinct 70B layer seeds resident in HBM; a step decodes all of "
                         "them (80: every layer of the 70B model)")
    ap.add_argument("--chunk-bytes", type=int, default=65536)
    ap.add_argument("--lanes", type=int, default=64)
    ap.add_argument("--threads", type=int, default=int(os.environ.get("OMP_NUM_THREADS", "16")))
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--two-stream", action="store_true",
                    help="also time the same steps with consecutive launches issued "
                         "alternately on two streams (supplementary; launches overlap, so a "
                         "kernel trace of such a run no longer gives per-launch durations)")
    ap.add_argument("--no-two-stream", action="store_true", help=argparse.SUPPRESS)
    ap.add_argument("--tile", default="", help="ROWSxCOLS 2-D tiles, e.g. 128x256 (default: "
                    "flat chunks of --chunk-bytes)")
    ap.add_argument("--codebook", choices=["tensor", "layer"], default="tensor")
    ap.add_argument("--nibbles-as-bytes", action="store_true",
                    help="code 4-bit tensors (int4, fp4 codes) by their packed bytes, two "
                         "nibbles per symbol, instead of one symbol per nibble")
    ap.add_argument("--sweep", action="store_true",
                    help="one bf16 decoder layer of each model family of the paper (1.5B to "
                         "405B parameters), drawn on the GPU and compressed with the device "
                         "encoder: one JSON line per model")
    ap.add_argument("--encode", action="store_true",
                    help="time the device encoder (wc_encode_device) on the resident 70B "
                         "layer instead of the decode")
    ap.add_argument("--gemv", type=int, default=0, metavar="M",
                    help="time the fused decode-GEMM y += x W^T (x: M rows, 1..4096) over a "
                         "bf16 layer (--gemv-layer) instead of the decode, next to the same "
                         "product unfused (wc_decode, then torch.matmul) and uncompressed "
                         "(torch.matmul)")
    ap.add_argument("--gemv-rows", type=int, choices=[64, 32, 16], default=0,
                    help="tile rows of the fused GEMM: 64 (VALU dot products for M <= 5, "
                         "matrix cores above), 32 or 16 (matrix cores); default 16 for "
                         "M <= 16, else 64")
    ap.add_argument("--gemv-layer", choices=["70b", "8b"], default="70b",
                    help="the bf16 layer of --gemv: the Llama-3-70B layer (default) or the "
                         "Llama-3-8B layer, the latter rotated over resident copies")
    ap.add_argument("--gemm-i8", type=int, default=0, metavar="M",
                    help="time the fused int8 decode-GEMM (W8A8: int8 x, int32 y, "
                         "v_mfma_i32_16x16x64_i8; M rows, 1..64) over the int8 projections of "
                         "the 8B W8 layer in 16 x 2048 tiles, next to the same product unfused "
                         "and uncompressed (torch._int_mm)")
    ap.add_argument("--gemv-fp8", type=int, default=0, metavar="M",
                    help="time the fused decode-GEMM on fp8 weights (bf16 x, fp32 y; "
                         "M rows, 1..64) over the fp8 projections of the 8B fp8 layer in "
                         "16 x 2048 tiles, next to the same product unfused and on the "
                         "weights kept as bf16")
    ap.add_argument("--gemv-mx", type=int, default=0, metavar="M",
                    help="time the fused decode-GEMM on MXFP4 weights (wc_gemv_mx: e2m1 codes "
                         "with e8m0 scales per 32, bf16 x, fp32 y; M rows, 1..64) over the "
                         "seven projections of the 8B MXFP4 layer in 16 x 2048 tiles, next to "
                         "the same product unfused and on the weights kept as bf16")
    ap.add_argument("--gemv-w4", type=int, default=0, metavar="M",
                    help="time the fused decode-GEMM on group-quantised int4 weights "
                         "(wc_gemv_w4: codes as bytes, fp16 scales per 128, zero points; "
                         "bf16 x, fp32 y; M rows, 1..64) over the seven projections of the "
                         "8B AWQ-style layer (--w4-signed: the symmetric int4 layer) in "
                         "16 x 1024-byte tiles, next to the same product unfused and on the "
                         "weights kept as bf16")
    ap.add_argument("--w4-signed", action="store_true",
                    help="--gemv-w4 on the two's-complement int4 layer (no zero points)")
    ap.add_argument("--w4-nibbles", action="store_true",
                    help="--gemv-w4 with the codes as nibble symbols (WC_U4) instead of bytes")
    ap.add_argument("--mx-bytes", action="store_true",
                    help="--gemv-mx: code the packed e2m1 bytes as byte symbols (WC_U8) "
                         "instead of nibble symbols: half the decode steps")
    ap.add_argument("--fp8-format", choices=["e4m3", "e5m2"], default="e4m3",
                    help="fp8 format of --gemv-fp8 (the llama3-8b-layer-fp8-e4m3 or "
                         "-fp8-e5m2 workload)")
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
    if args.gemv:
        return gemv_bench(args, dev)
    if args.gemm_i8:
        return gemm_i8_bench(args, dev)
    if args.gemv_fp8:
        return gemv_fp8_bench(args, dev)
    if args.gemv_mx:
        return gemv_mx_bench(args, dev)
    if args.gemv_w4:
        return gemv_w4_bench(args, dev)
    if args.encode:
        return encode_bench(args, dev)
    if args.sweep:
        return sweep_bench(args, dev)
    cfg = WORKLOADS[args.workload]
    big = cfg == 5
    tile = tuple(int(v) for v in args.tile.lower().split("x")) if args.tile else (0, 0)
    shaped = lambda t, d, shape: (t, d, shape if len(shape) == 2 else None)  # noqa: E731

    # --- setup: draw, encode, upload, verify ---------------------------------
    # The 70B workload keeps `--layers` distinct layer blobs and a step decodes
    # every one of them, back to back (80 layers: the sustained run over a whole
    # model's layers); the others keep copies of one blob and a step decodes one
    # copy.  Launch g decodes resident blob g mod n_res.
    err = torch.zeros(1, dtype=torch.int32, device=dev)
    blobs, dblobs, sets = [], [], []
    keep_orig = {}
    comp = cpu = cpu_all = None
    t_setup = time.perf_counter()

    def check(blob, dblob, outs, originals, what):
        wc.decode_torch(blob, dblob, outs=outs, err=err)
        torch.cuda.synchronize()
        if int(err.item()) != 0:
            raise RuntimeError(f"{what}: device errors {wc.describe_errors(int(err.item()))}")
        for orig, out in zip(originals, outs):
            if not torch.equal(orig.reshape(-1).view(torch.uint8), out[:orig.numel() * orig.element_size()]):
                raise RuntimeError(f"{what}: decoded bytes differ from the original")

    def first_blob(typed_host):
        nonlocal comp, cpu, cpu_all
        comp = compression_stats(blobs[0], typed_host)
        if not args.no_cpu_baseline:
            log("cpu baseline: oracle decode, one core, then all cores ...")
            cpu, cpu_all = oracle_baseline(blobs[0], [h for _, h in typed_host], args.workload)
            log(f"cpu baseline: {cpu['value']} GB/s on one core ({cpu['seconds']} s), "
                f"{cpu_all['value']} GB/s on {cpu_all['cores']} cores")

    if big:
        n_res = max(1, args.layers)
        per_step = n_res
        last = {(n_res - j) % n_res for j in (1, 2)}
        for layer in range(n_res):
            t0 = time.perf_counter()
            tens = synth.config_torch_device(5, layer, device="cuda")
            host = [("bf16", t.cpu().numpy()) for _, t, _ in tens]
            blob = wc.encode([shaped(dt, h, shape) for (dt, h), (_, _, shape) in zip(host, tens)],
                             chunk_bytes=args.chunk_bytes, lanes=args.lanes,
                             threads=args.threads, tile=tile, codebook=args.codebook)
            blobs.append(blob)
            dblobs.append(wc.to_device(blob, dev))
            if len(sets) == 0:
                sets = [[torch.empty(n, dtype=torch.uint8, device=dev) for n in blob.out_bytes]
                        for _ in range(2)]
            check(blob, dblobs[-1], sets[0], [o for _, o, _ in tens], f"layer {layer}")
            if layer in last:
                keep_orig[layer] = [o for _, o, _ in tens]
            if layer == 0:
                first_blob(host)
            del tens, host
            log(f"layer {layer + 1}/{n_res}: {blob.size / 1e9:.3f} GB compressed, "
                f"{sum(blob.out_bytes) / 1e9:.3f} GB decoded, verified, "
                f"{time.perf_counter() - t0:.1f} s")
        out_sets = lambda g: sets[g % 2]          # noqa: E731
        origs = lambda g: keep_orig[g % n_res]    # noqa: E731
    else:
        per_step = 1
        tens = synth.config(cfg)
        # --nibbles-as-bytes: a packed 4-bit tensor becomes a byte tensor of half
        # the columns (two nibbles per symbol); the decoded bytes are the same
        nib = lambda t: args.nibbles_as_bytes and t.dtype in ("u4", "fp4_e2m1")  # noqa: E731
        sym = lambda t: "u8" if nib(t) else t.dtype  # noqa: E731
        shp = lambda t: (t.shape[0], t.shape[1] // 2) if nib(t) and len(t.shape) == 2 else t.shape  # noqa: E731
        host = [(sym(t), t.data) for t in tens]
        blob = wc.encode([shaped(sym(t), t.data, shp(t)) for t in tens],
                         chunk_bytes=args.chunk_bytes, lanes=args.lanes,
                         threads=args.threads, tile=tile, codebook=args.codebook)
        per = blob.size + sum(blob.out_bytes)
        n_res = max(2, -(-ROTATE_BYTES // per))
        dev_orig = [torch.from_numpy(np.ascontiguousarray(h).view(np.uint8).reshape(-1)).to(dev)
                    for _, h in host]
        for r in range(n_res):
            blobs.append(blob)
            dblobs.append(wc.to_device(blob, dev))
            sets.append([torch.empty(n, dtype=torch.uint8, device=dev) for n in blob.out_bytes])
            check(blob, dblobs[-1], sets[-1], dev_orig, f"copy {r}")
        first_blob(host)
        log(f"{args.workload}: {blob.size / 1e6:.1f} MB compressed, "
            f"{sum(blob.out_bytes) / 1e6:.1f} MB decoded, {n_res} resident copies, verified")
        out_sets = lambda g: sets[g % n_res]      # noqa: E731
        origs = lambda g: dev_orig                # noqa: E731
        del tens
    torch.cuda.empty_cache()
    setup_s = time.perf_counter() - t_setup
    out_per_launch = sum(blobs[0].out_bytes)
    in_per_launch = float(np.mean([b.size for b in blobs]))
    out_per_step = per_step * out_per_launch
    stream = torch.cuda.current_stream(dev)

    # --- ceilings: the same byte mix through a plain streaming kernel ---------
    # wc_stream reads the compressed bytes of one launch once and writes its
    # decoded bytes once (non-temporal stores), with no decoding in between;
    # the best of a few grid sizes.  Beside it, torch's device-to-device copy
    # of 512 MiB (twice the Infinity Cache).
    # Launches rotate over enough (source, destination) pairs (>= 1 GiB) that
    # none finds its bytes in the Infinity Cache, as the decode launches do.
    n_in = int(in_per_launch) // 16 * 16
    n_out = out_per_launch // 16 * 16
    n_cp = 1 if big else rotation_copies(n_in + n_out)
    pairs = []
    for _ in range(n_cp):
        src = torch.empty(n_in, dtype=torch.uint8, device=dev)
        src.random_(0, 256)
        pairs.append((src, torch.empty(n_out, dtype=torch.uint8, device=dev)))
    sweep = {}
    for blocks in (8192, 16384, 32768, 65536, 131072):
        def sl(k):
            src, dst = pairs[k % n_cp]
            return wc.stream_bytes(src.data_ptr(), n_in, dst.data_ptr(), n_out, blocks,
                                   stream.cuda_stream)
        for k in range(2):
            rd = sl(k)
        sev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in range(10)]
        for k, (e0, e1) in enumerate(sev):
            e0.record(stream)
            sl(k)
            e1.record(stream)
        torch.cuda.synchronize()
        med = float(np.median([e0.elapsed_time(e1) for e0, e1 in sev])) / 1e3
        sweep[blocks] = ((rd + n_out) / med / 1e9, med, rd)
    best = max(sweep, key=lambda k: sweep[k][0])
    ceiling = {"kernel": "wc_stream_kernel", "GBps": round(sweep[best][0], 1),
               "frac": round(sweep[best][0] / HBM_PEAK_GBPS, 4),
               "read_bytes": sweep[best][2], "write_bytes": n_out,
               "median_launch_us": round(sweep[best][1] * 1e6, 2),
               "blocks": best, "copies_resident": n_cp,
               "sweep_GBps": {str(k): round(v[0], 1) for k, v in sweep.items()},
               "timing": "median of 10 event-timed launches per grid size; best grid"}
    del pairs
    csrc = torch.empty(512 << 20, dtype=torch.uint8, device=dev)
    cdst = torch.empty_like(csrc)
    for _ in range(3):
        cdst.copy_(csrc)
    torch.cuda.synchronize()
    c0, c1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    c0.record()
    for _ in range(10):
        cdst.copy_(csrc)
    c1.record()
    torch.cuda.synchronize()
    copy_gbps = 10 * 2 * csrc.numel() / (c0.elapsed_time(c1) / 1e3) / 1e9
    del csrc, cdst
    torch.cuda.empty_cache()

    # --- timed decode ---------------------------------------------------------
    err.zero_()

    def launch(g, s):
        r = g % n_res
        wc.decode(blobs[r], dblobs[r].data_ptr(), [o.data_ptr() for o in out_sets(g)],
                  s.cuda_stream, err.data_ptr())

    W, K = args.warmup, args.steps
    for g in range(W * per_step):
        launch(g, stream)
    torch.cuda.synchronize()
    G = K * per_step
    # one event between consecutive launches: launch j runs between ev[j] and ev[j + 1]
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(G + 1)]
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record(stream)
    for j in range(G):
        ev[j].record(stream)
        launch(W * per_step + j, stream)
    ev[G].record(stream)
    end.record(stream)
    torch.cuda.synchronize()
    total_ms = start.elapsed_time(end)
    launch_ms = [ev[j].elapsed_time(ev[j + 1]) for j in range(G)]

    def verify_last(what):
        if int(err.item()) != 0:
            raise RuntimeError(f"device errors during {what}: "
                               f"{wc.describe_errors(int(err.item()))}")
        for j in (1, 2):
            g = (W + K) * per_step - j
            if g < W * per_step:
                continue
            for o, r in zip(out_sets(g), origs(g)):
                if not torch.equal(o[:r.numel() * r.element_size()], r.reshape(-1).view(torch.uint8)):
                    raise RuntimeError(f"{what}: decode output differs from the original")

    verify_last("the timed decode")

    # --- the same steps on two streams (supplementary) --------------------------
    two = None
    if args.two_stream:
        streams = [torch.cuda.Stream(dev), torch.cuda.Stream(dev)]
        for g in range(W * per_step):
            launch(g, streams[g % 2])
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for j in range(G):
            g = W * per_step + j
            launch(g, streams[g % 2])
        torch.cuda.synchronize()
        dt2 = time.perf_counter() - t0
        verify_last("the two-stream decode")
        two = {"value": round(K * out_per_step / dt2 / 1e9, 2), "unit": "GB/s",
               "ms_per_step": round(dt2 / K * 1e3, 4),
               "timing": "host clock around the K steps with consecutive launches issued "
                         "alternately on two streams"}

    value = K * out_per_step / (total_ms / 1e3) / 1e9
    med_launch_s = float(np.median(launch_ms)) / 1e3
    mean_launch_s = float(np.mean(launch_ms)) / 1e3
    achieved = (in_per_launch + out_per_launch) / med_launch_s / 1e9
    config = {"workload": args.workload, "tensors_per_launch": len(blobs[0].out_bytes),
              "launches_per_step": per_step,
              "decoded_bytes_per_step": out_per_step,
              "compressed_bytes_per_step": int(per_step * in_per_launch),
              "chunk_bytes": args.chunk_bytes, "lanes": args.lanes, "parallelism": "single-gpu"}
    if args.tile:
        config["tile"] = args.tile
    if args.codebook != "tensor":
        config["codebook"] = args.codebook
    if args.nibbles_as_bytes:
        config["symbols"] = "4-bit tensors coded by packed bytes (two nibbles per symbol)"
    if big:
        config["layers_resident"] = n_res
        config["step"] = f"one wc_decode launch per resident layer, {n_res} back to back"
    else:
        config["copies_resident"] = n_res
        config["step"] = "one wc_decode launch of one resident copy"
    kname = decode_kernel_for([blobs[0].dtype(t) for t in range(blobs[0].n_tensors)],
                              blobs[0].n_chunks, args.lanes, bool(args.tile))
    line = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": W,
        "ms_per_step": round(total_ms / K, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u32",
        "data": "synthetic",
        "config": config,
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBPS, 4),
                     "traffic": counted_traffic(args.workload, args.chunk_bytes, args.lanes,
                                                bool(args.tile) or args.codebook != "tensor",
                                                kname),
                     "kernel": kname,
                     "median_launch_us": round(med_launch_s * 1e6, 2),
                     "mean_launch_us": round(mean_launch_s * 1e6, 2),
                     "launches_timed": G,
                     "algorithmic_bytes_per_launch": int(in_per_launch + out_per_launch),
                     "of_ceiling": round(achieved / ceiling["GBps"], 4)},
        "hbm_pct": round(100 * achieved / HBM_PEAK_GBPS, 2),
        "ceiling": ceiling,
        "d2d_copy_GBps": round(copy_gbps, 1),
        "two_stream": two,
        "compression": comp,
        "cpu_baseline": cpu,
        "cpu_baseline_all_cores": cpu_all,
        "setup_s": round(setup_s, 1),
    }
    print(json.dumps(line), flush=True)
    return 0


def gemv_bench(args, dev) -> int:
    """Fused decode-GEMM over the seven projections of one bf16 layer: the 70B
    layer (one copy, 1.7 GB of weights), or with --gemv-layer 8b the 8B layer,
    whose variants rotate over resident copies (>= 1 GiB each)."""
    import numpy as np
    import torch

    from paper_2606_15789_amd import synth, wc
    M = args.gemv
    rows = args.gemv_rows or (16 if M <= 16 else 64)
    if not 1 <= M <= (4096 if rows == 64 else 64):
        print("--gemv takes 1..4096 rows of activations on 64-row tiles, 1..64 on 32- or "
              "16-row tiles", file=sys.stderr)
        return 2
    # 64 KiB tiles: 64 x 512 (a lane per W row, VALU dot products), 32 x 1024 or
    # 16 x 2048 (a wave row per MFMA operand)
    tile = {64: (64, 512), 32: (32, 1024), 16: (16, 2048)}[rows]
    t0 = time.perf_counter()
    if args.gemv_layer == "8b":
        workload = "llama3-8b-layer-bf16"
        tens = synth.layer_torch_device(synth.LLAMA3_8B, 0.02, 1, 0, device="cuda")
    else:
        workload = "llama3-70b-layer-bf16"
        tens = synth.config_torch_device(5, 0, device="cuda")
    shapes = [shape for _, _, shape in tens]
    host = [t.cpu().numpy() for _, t, _ in tens]
    blob = wc.encode([("bf16", h, shp) for h, shp in zip(host, shapes)], lanes=64, tile=tile,
                     tile_order=1, threads=args.threads)
    del host
    dblob = wc.to_device(blob, dev)
    W = [t.view(torch.bfloat16).reshape(shp) for _, t, shp in tens]
    gen = torch.Generator(device=dev)
    gen.manual_seed(12345)
    xs = [torch.randn(M, shp[1], generator=gen, device=dev).to(torch.bfloat16) for shp in shapes]
    ys = [torch.zeros(M, shp[0], dtype=torch.float32, device=dev) for shp in shapes]
    err = torch.zeros(1, dtype=torch.int32, device=dev)
    stream = torch.cuda.current_stream(dev)

    # wc_gemm: wc_gemv up to 64 rows; above, x is packed into the workspace
    # (inside every timed call) and the weights are decoded once per 256 rows
    need = wc.gemm_workspace_bytes(blob, list(range(len(W))), [x.data_ptr() for x in xs], M)
    ws = torch.empty(max(need, 256), dtype=torch.uint8, device=dev)

    def fused(d=dblob):
        # one launch per tile height for the seven projections (plus the x packing)
        wc.gemm(blob, d.data_ptr(), list(range(len(W))), [x.data_ptr() for x in xs], M,
                [y.data_ptr() for y in ys], ws.data_ptr(), ws.numel(), stream.cuda_stream,
                err.data_ptr())

    # correctness: y against torch's fp32 product of the same bf16 values,
    # within the fp32 summation bound K * 2^-23 * sum |x w|
    fused()
    torch.cuda.synchronize()
    if int(err.item()):
        raise RuntimeError(f"device errors: {wc.describe_errors(int(err.item()))}")
    for t, (w, x, y) in enumerate(zip(W, xs, ys)):
        ref = x.float() @ w.float().t()
        bound = x.float().abs() @ w.float().abs().t()
        if torch.any((y - ref).abs() > w.shape[1] * 2.0 ** -23 * bound + 1e-30):
            raise RuntimeError(f"fused GEMM tensor {t} outside the fp32 summation bound")
    setup_s = time.perf_counter() - t0

    # the unfused path decodes a byte-run blob of the same layer (the decode's
    # fastest layout: 1 KiB rows) into memory, then multiplies
    flat = wc.encode([("bf16", w.view(torch.uint8).reshape(-1).cpu().numpy()) for w in W],
                     lanes=64, threads=args.threads)
    dflat = wc.to_device(flat, dev)
    outs = [torch.empty(n, dtype=torch.uint8, device=dev) for n in flat.out_bytes]

    # the 70B layer is well past the 256 MB Infinity Cache in one copy; the 8B
    # layer's variants rotate over resident copies of their operands
    if args.gemv_layer == "8b":
        n_f = rotation_copies(blob.size)
        n_u = rotation_copies(flat.size + sum(flat.out_bytes))
        n_p = rotation_copies(sum(w.numel() * 2 for w in W))
    else:
        n_f = n_u = n_p = 1
    dblobs = [dblob] + [dblob.clone() for _ in range(n_f - 1)]
    dflats = [dflat] + [dflat.clone() for _ in range(n_u - 1)]
    outss = [outs] + [[torch.empty_like(o) for o in outs] for _ in range(n_u - 1)]
    Ws = [W] + [[w.clone() for w in W] for _ in range(n_p - 1)]

    def fused_k(k):
        fused(dblobs[k % n_f])

    def unfused(k):
        o_k = outss[k % n_u]
        wc.decode(flat, dflats[k % n_u].data_ptr(), [o.data_ptr() for o in o_k],
                  stream.cuda_stream, err.data_ptr())
        for t, (o, x, shp) in enumerate(zip(o_k, xs, shapes)):
            torch.matmul(x, o.view(torch.bfloat16).view(shp).t())

    def uncompressed(k):
        for w, x in zip(Ws[k % n_p], xs):
            torch.matmul(x, w.t())

    s_fused, s_unfused, s_plain = (timed_rotating(f, args.warmup, args.steps, stream)
                                   for f in (fused_k, unfused, uncompressed))
    if int(err.item()):
        raise RuntimeError(f"device errors: {wc.describe_errors(int(err.item()))}")
    wbytes = sum(blob.out_bytes)
    alg = blob.size + sum(x.numel() * 2 for x in xs) + sum(2 * y.numel() * 4 for y in ys)
    achieved = alg / s_fused / 1e9
    flops = sum(2.0 * M * shp[0] * shp[1] for shp in shapes)
    tflops = flops / s_fused / 1e12
    shared = rows == 64 and M > 64
    # the bound: HBM below the ridge point (peak flops / peak bytes), MFMA above
    mfma_bound = flops / alg > MFMA_BF16_PEAK_TFLOPS * 1e12 / (HBM_PEAK_GBPS * 1e9)
    line = {
        "metric": METRIC + " [fused decode-GEMM]",
        "value": round(wbytes / s_fused / 1e9, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(s_fused * 1e3, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16 x bf16 -> fp32",
        "data": "synthetic",
        "config": {"workload": workload, "mode": "fused-gemv", "m": M,
                   "tile": f"{tile[0]}x{tile[1]}", "tile_order": "column-blocks",
                   "product": ("v_dot2_f32_bf16" if rows == 64 and M <= 5 else
                               "v_mfma_f32_16x16x32_bf16" if rows == 16 else
                               "v_mfma_f32_32x32x16_bf16"),
                   "decoded_once_per": ("256 rows of x (operands shared through LDS)"
                                        if shared else "call"),
                   "lanes": 64, "weight_bytes_per_step": wbytes,
                   "compressed_bytes_per_step": blob.size,
                   "copies_resident": {"fused": n_f, "unfused": n_u, "uncompressed": n_p},
                   "parallelism": "single-gpu"},
        "roofline": ({"bound": "mfma", "achieved": round(tflops, 1),
                      "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                      "frac": round(tflops / MFMA_BF16_PEAK_TFLOPS, 4), "traffic": None}
                     if mfma_bound else
                     {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS,
                      "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBPS, 4),
                      "traffic": None})
                    | {"kernel": ("wc_gemm_kernel" if shared else
                                  gemv_kernel_for("bf16", blob.n_chunks, M) if rows == 16 else
                                  "wc_gemv_kernel"),
                       "mean_step_us": round(s_fused * 1e6, 2),
                       "algorithmic_bytes_per_step": int(alg), "flops_per_step": flops,
                       "hbm_frac": round(achieved / HBM_PEAK_GBPS, 4),
                       "mfma_frac": round(tflops / MFMA_BF16_PEAK_TFLOPS, 4)},
        "unfused": {"value": round(wbytes / s_unfused / 1e9, 2), "unit": "GB/s",
                    "ms_per_step": round(s_unfused * 1e3, 4),
                    "what": "wc_decode of the layer (64 KiB byte-run chunks) into memory, then "
                            "torch.matmul per tensor"},
        "uncompressed": {"value": round(wbytes / s_plain / 1e9, 2), "unit": "GB/s",
                         "ms_per_step": round(s_plain * 1e3, 4),
                         "what": "torch.matmul on the bf16 weights"},
        "setup_s": round(setup_s, 1),
    }
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = oracle_gemv_baseline(blob, W[0].cpu().view(torch.int16).numpy().view(np.uint16),
                                                    M, wbytes)
    print(json.dumps(line), flush=True)
    return 0


def gemm_i8_bench(args, dev) -> int:
    """Fused int8 decode-GEMM (W8A8) over the seven int8 projections of the 8B
    W8 layer: exact int32 y, checked against an fp64 product (exact here)."""
    import numpy as np
    import torch

    from paper_2606_15789_amd import synth, wc
    M = args.gemm_i8
    if not 1 <= M <= 64:
        print("--gemm-i8 takes 1..64 rows of activations", file=sys.stderr)
        return 2
    tile = (16, 2048)
    t0 = time.perf_counter()
    ts = [t for t in synth.config(4) if t.dtype == "u8" and len(t.shape) == 2]
    shapes = [t.shape for t in ts]
    blob = wc.encode([(t.dtype, t.data, t.shape) for t in ts], lanes=64, tile=tile,
                     tile_order=1, threads=args.threads)
    dblob = wc.to_device(blob, dev)
    W = [torch.from_numpy(np.ascontiguousarray(t.data).view(np.int8).reshape(t.shape)).to(dev)
         for t in ts]
    gen = torch.Generator(device=dev)
    gen.manual_seed(54321)
    xs = [torch.randint(-127, 128, (M, shp[1]), generator=gen, device=dev, dtype=torch.int8)
          for shp in shapes]
    ys = [torch.zeros(M, shp[0], dtype=torch.int32, device=dev) for shp in shapes]
    err = torch.zeros(1, dtype=torch.int32, device=dev)
    stream = torch.cuda.current_stream(dev)

    def fused():
        wc.gemm_i8(blob, dblob.data_ptr(), list(range(len(W))), [x.data_ptr() for x in xs], M,
                   [y.data_ptr() for y in ys], stream.cuda_stream, err.data_ptr())

    fused()
    torch.cuda.synchronize()
    if int(err.item()):
        raise RuntimeError(f"device errors: {wc.describe_errors(int(err.item()))}")
    for t, (w, x, y) in enumerate(zip(W, xs, ys)):
        # |y| < 2^30: the fp64 product is exact
        if not torch.equal(y.double(), x.double() @ w.double().t()):
            raise RuntimeError(f"int8 fused GEMM tensor {t} differs from the exact product")
    setup_s = time.perf_counter() - t0

    # uncompressed int8 GEMM: torch._int_mm (hipBLASLt) where it takes the shape
    def int_mm(x, w):
        return torch._int_mm(x, w.t())
    try:
        xp = torch.zeros(max(M, 32), shapes[0][1], dtype=torch.int8, device=dev)
        int_mm(xp, W[0])
        xs_mm = [torch.zeros(max(M, 32), shp[1], dtype=torch.int8, device=dev) for shp in shapes]
        for xm, x in zip(xs_mm, xs):
            xm[:M].copy_(x)
        base_what = ("torch._int_mm (int8 x int8 -> int32) on the int8 weights" +
                     (f", x padded to {max(M, 32)} rows (its smallest M)" if M < 32 else ""))
        mm = int_mm
    except RuntimeError:
        xs_mm = [x.to(torch.bfloat16) for x in xs]
        Wb = [w.to(torch.bfloat16) for w in W]
        base_what = "torch.matmul in bf16 on the int8 weights (no int8 GEMM for this shape)"
        mm = None

    flat = wc.encode([("u8", np.ascontiguousarray(t.data).reshape(-1)) for t in ts], lanes=64,
                     threads=args.threads)
    dflat = wc.to_device(flat, dev)
    outs = [torch.empty(n, dtype=torch.uint8, device=dev) for n in flat.out_bytes]

    def product(i, w):
        return mm(xs_mm[i], w) if mm else torch.matmul(xs_mm[i], w.t())

    # every variant rotates over resident copies of its weights (>= 1 GiB)
    n_f = rotation_copies(blob.size)
    dblobs = [dblob] + [dblob.clone() for _ in range(n_f - 1)]
    n_u = rotation_copies(flat.size + sum(flat.out_bytes))
    dflats = [dflat] + [dflat.clone() for _ in range(n_u - 1)]
    outss = [outs] + [[torch.empty_like(o) for o in outs] for _ in range(n_u - 1)]
    Wp = W if mm else Wb
    n_p = rotation_copies(sum(w.numel() * w.element_size() for w in Wp))
    Wps = [Wp] + [[w.clone() for w in Wp] for _ in range(n_p - 1)]

    def fused_k(k):
        wc.gemm_i8(blob, dblobs[k % n_f].data_ptr(), list(range(len(W))),
                   [x.data_ptr() for x in xs], M, [y.data_ptr() for y in ys], stream.cuda_stream,
                   err.data_ptr())

    def unfused(k):
        o_k = outss[k % n_u]
        wc.decode(flat, dflats[k % n_u].data_ptr(), [o.data_ptr() for o in o_k],
                  stream.cuda_stream, err.data_ptr())
        for i, (o, shp) in enumerate(zip(o_k, shapes)):
            w = o.view(torch.int8).view(shp)
            product(i, w if mm else w.to(torch.bfloat16))

    def uncompressed(k):
        for i, w in enumerate(Wps[k % n_p]):
            product(i, w)

    s_fused, s_unfused, s_plain = (timed_rotating(f, args.warmup, args.steps, stream)
                                   for f in (fused_k, unfused, uncompressed))
    if int(err.item()):
        raise RuntimeError(f"device errors: {wc.describe_errors(int(err.item()))}")
    wbytes = sum(blob.out_bytes)
    alg = blob.size + sum(x.numel() for x in xs) + sum(2 * y.numel() * 4 for y in ys)
    achieved = alg / s_fused / 1e9
    line = {
        "metric": METRIC + " [fused int8 decode-GEMM]",
        "value": round(wbytes / s_fused / 1e9, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(s_fused * 1e3, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int8 x int8 -> int32",
        "data": "synthetic",
        "config": {"workload": "llama3-8b-layer-int8", "mode": "fused-gemm-i8", "m": M,
                   "tile": f"{tile[0]}x{tile[1]}", "tile_order": "column-blocks",
                   "product": "v_mfma_i32_16x16x64_i8", "lanes": 64,
                   "weight_bytes_per_step": wbytes, "compressed_bytes_per_step": blob.size,
                   "copies_resident": {"fused": n_f, "unfused": n_u, "uncompressed": n_p},
                   "parallelism": "single-gpu"},
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBPS, 4), "traffic": None,
                     "kernel": gemv_kernel_for("int8", blob.n_chunks, M),
                     "mean_step_us": round(s_fused * 1e6, 2),
                     "algorithmic_bytes_per_step": int(alg)},
        "unfused": {"value": round(wbytes / s_unfused / 1e9, 2), "unit": "GB/s",
                    "ms_per_step": round(s_unfused * 1e3, 4),
                    "what": "wc_decode of the weights (64 KiB byte-run chunks) into memory, then "
                            + base_what},
        "uncompressed": {"value": round(wbytes / s_plain / 1e9, 2), "unit": "GB/s",
                         "ms_per_step": round(s_plain * 1e3, 4), "what": base_what},
        "setup_s": round(setup_s, 1),
    }
    print(json.dumps(line), flush=True)
    return 0


def gemv_fp8_bench(args, dev) -> int:
    """Fused decode-GEMM over the seven fp8 (e4m3 or e5m2) projections of the 8B
    fp8 layer (bf16 x, fp32 y), checked against torch's fp32 product of the
    same values."""
    import numpy as np
    import torch

    from paper_2606_15789_amd import synth, wc
    M = args.gemv_fp8
    if not 1 <= M <= 64:
        print("--gemv-fp8 takes 1..64 rows of activations", file=sys.stderr)
        return 2
    fmt = args.fp8_format
    dtype = "fp8_" + fmt
    tdt = torch.float8_e4m3fn if fmt == "e4m3" else torch.float8_e5m2
    workload = "llama3-8b-layer-fp8-" + fmt
    tile = (16, 2048)
    t0 = time.perf_counter()
    ts = [t for t in synth.config(WORKLOADS[workload]) if t.dtype == dtype and len(t.shape) == 2]
    shapes = [t.shape for t in ts]
    blob = wc.encode([(t.dtype, t.data, t.shape) for t in ts], lanes=64, tile=tile,
                     tile_order=1, threads=args.threads)
    dblob = wc.to_device(blob, dev)
    W8 = [torch.from_numpy(np.ascontiguousarray(t.data).reshape(t.shape)).to(dev) for t in ts]
    Wb = [w.view(tdt).to(torch.bfloat16) for w in W8]   # exact
    gen = torch.Generator(device=dev)
    gen.manual_seed(24680)
    xs = [torch.randn(M, shp[1], generator=gen, device=dev).to(torch.bfloat16) for shp in shapes]
    ys = [torch.zeros(M, shp[0], dtype=torch.float32, device=dev) for shp in shapes]
    err = torch.zeros(1, dtype=torch.int32, device=dev)
    stream = torch.cuda.current_stream(dev)

    def fused():
        wc.gemv(blob, dblob.data_ptr(), list(range(len(ts))), [x.data_ptr() for x in xs], M,
                [y.data_ptr() for y in ys], stream.cuda_stream, err.data_ptr())

    fused()
    torch.cuda.synchronize()
    if int(err.item()):
        raise RuntimeError(f"device errors: {wc.describe_errors(int(err.item()))}")
    for t, (w, x, y) in enumerate(zip(Wb, xs, ys)):
        ref = x.float() @ w.float().t()
        bound = x.float().abs() @ w.float().abs().t()
        if torch.any((y - ref).abs() > w.shape[1] * 2.0 ** -23 * bound + 1e-30):
            raise RuntimeError(f"fp8 fused GEMM tensor {t} outside the fp32 summation bound")
    setup_s = time.perf_counter() - t0

    flat = wc.encode([(dtype, np.ascontiguousarray(t.data).reshape(-1)) for t in ts],
                     lanes=64, threads=args.threads)
    dflat = wc.to_device(flat, dev)
    outs = [torch.empty(n, dtype=torch.uint8, device=dev) for n in flat.out_bytes]

    # every variant rotates over resident copies of its weights (>= 1 GiB)
    n_f = rotation_copies(blob.size)
    dblobs = [dblob] + [dblob.clone() for _ in range(n_f - 1)]
    n_u = rotation_copies(flat.size + sum(flat.out_bytes))
    dflats = [dflat] + [dflat.clone() for _ in range(n_u - 1)]
    outss = [outs] + [[torch.empty_like(o) for o in outs] for _ in range(n_u - 1)]
    n_p = rotation_copies(sum(w.numel() * 2 for w in Wb))
    Wbs = [Wb] + [[w.clone() for w in Wb] for _ in range(n_p - 1)]

    def fused_k(k):
        wc.gemv(blob, dblobs[k % n_f].data_ptr(), list(range(len(ts))),
                [x.data_ptr() for x in xs], M, [y.data_ptr() for y in ys], stream.cuda_stream,
                err.data_ptr())

    def unfused(k):
        o_k = outss[k % n_u]
        wc.decode(flat, dflats[k % n_u].data_ptr(), [o.data_ptr() for o in o_k],
                  stream.cuda_stream, err.data_ptr())
        for o, x, shp in zip(o_k, xs, shapes):
            w = o.view(tdt).view(shp).to(torch.bfloat16)
            torch.matmul(x, w.t())

    def uncompressed(k):
        for w, x in zip(Wbs[k % n_p], xs):
            torch.matmul(x, w.t())

    s_fused, s_unfused, s_plain = (timed_rotating(f, args.warmup, args.steps, stream)
                                   for f in (fused_k, unfused, uncompressed))
    if int(err.item()):
        raise RuntimeError(f"device errors: {wc.describe_errors(int(err.item()))}")
    wbytes = sum(blob.out_bytes)
    alg = blob.size + sum(x.numel() * 2 for x in xs) + sum(2 * y.numel() * 4 for y in ys)
    achieved = alg / s_fused / 1e9
    line = {
        "metric": METRIC + " [fused fp8 decode-GEMM]",
        "value": round(wbytes / s_fused / 1e9, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(s_fused * 1e3, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": f"fp8 {fmt} (as bf16) x bf16 -> fp32",
        "data": "synthetic",
        "config": {"workload": workload, "mode": "fused-gemv-fp8", "m": M,
                   "tile": f"{tile[0]}x{tile[1]}", "tile_order": "column-blocks",
                   "product": ("v_cvt_scalef32_pk_bf16_" + ("fp8" if fmt == "e4m3" else "bf8") +
                               " + v_mfma_f32_16x16x32_bf16"),
                   "lanes": 64, "weight_bytes_per_step": wbytes,
                   "compressed_bytes_per_step": blob.size,
                   "copies_resident": {"fused": n_f, "unfused": n_u, "uncompressed": n_p},
                   "parallelism": "single-gpu"},
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBPS, 4), "traffic": None,
                     "kernel": gemv_kernel_for(fmt, blob.n_chunks, M),
                     "mean_step_us": round(s_fused * 1e6, 2),
                     "algorithmic_bytes_per_step": int(alg)},
        "unfused": {"value": round(wbytes / s_unfused / 1e9, 2), "unit": "GB/s",
                    "ms_per_step": round(s_unfused * 1e3, 4),
                    "what": "wc_decode of the fp8 weights (64 KiB byte-run chunks), torch "
                            "conversion to bf16, torch.matmul per tensor"},
        "uncompressed": {"value": round(wbytes / s_plain / 1e9, 2), "unit": "GB/s",
                         "ms_per_step": round(s_plain * 1e3, 4),
                         "what": "torch.matmul on the weights kept resident as bf16 (2x the "
                                 "fp8 bytes)"},
        "setup_s": round(setup_s, 1),
    }
    print(json.dumps(line), flush=True)
    return 0


def gemv_mx_bench(args, dev) -> int:
    """Fused decode-GEMM over the seven MXFP4 projections of the 8B MXFP4 layer
    (e2m1 codes in the blob, e8m0 scales decoded once, bf16 x, fp32 y), checked
    against torch's fp32 product of the same values."""
    import numpy as np
    import torch

    from paper_2606_15789_amd import synth, wc
    M = args.gemv_mx
    if not 1 <= M <= 64:
        print("--gemv-mx takes 1..64 rows of activations", file=sys.stderr)
        return 2
    workload = "llama3-8b-layer-mxfp4"
    tile = (16, 2048)
    t0 = time.perf_counter()
    ts = synth.config(WORKLOADS[workload])
    blocks = [t for t in ts if t.dtype == "fp4_e2m1"]
    scales = [t for t in ts if t.name.endswith(".scales")]
    shapes = [t.shape for t in blocks]
    if args.mx_bytes:
        blob = wc.encode([("u8", t.data, (t.shape[0], t.shape[1] // 2)) for t in blocks],
                         lanes=64, tile=(tile[0], tile[1] // 2), tile_order=1,
                         threads=args.threads)
    else:
        blob = wc.encode([(t.dtype, t.data, t.shape) for t in blocks], lanes=64, tile=tile,
                         tile_order=1, threads=args.threads)
    dblob = wc.to_device(blob, dev)
    dsc = [torch.from_numpy(np.ascontiguousarray(s.data).reshape(-1)).to(dev) for s in scales]
    lut = torch.tensor([0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0,
                        -0.0, -0.5, -1.0, -1.5, -2.0, -3.0, -4.0, -6.0],
                       dtype=torch.float32, device=dev)

    def dequant(packed, sc, shp):
        """bf16 weights of packed e2m1 codes and e8m0 scales (exact)."""
        p = packed.view(shp[0], shp[1] // 2)
        codes = torch.stack([p & 15, p >> 4], dim=2).reshape(shp).long()
        e = sc.view(shp[0], shp[1] // 32).int() - 127
        scale = torch.pow(2.0, e.float()).repeat_interleave(32, dim=1)
        return (lut[codes] * scale).to(torch.bfloat16)

    Wb = [dequant(torch.from_numpy(np.ascontiguousarray(t.data).reshape(-1)).to(dev), s, shp)
          for t, s, shp in zip(blocks, dsc, shapes)]
    gen = torch.Generator(device=dev)
    gen.manual_seed(13579)
    xs = [torch.randn(M, shp[1], generator=gen, device=dev).to(torch.bfloat16) for shp in shapes]
    ys = [torch.zeros(M, shp[0], dtype=torch.float32, device=dev) for shp in shapes]
    err = torch.zeros(1, dtype=torch.int32, device=dev)
    stream = torch.cuda.current_stream(dev)

    def fused():
        wc.gemv_mx(blob, dblob.data_ptr(), list(range(len(blocks))), [s.data_ptr() for s in dsc],
                   [x.data_ptr() for x in xs], M, [y.data_ptr() for y in ys],
                   stream.cuda_stream, err.data_ptr())

    fused()
    torch.cuda.synchronize()
    if int(err.item()):
        raise RuntimeError(f"device errors: {wc.describe_errors(int(err.item()))}")
    for t, (w, x, y) in enumerate(zip(Wb, xs, ys)):
        ref = x.float() @ w.float().t()
        bound = x.float().abs() @ w.float().abs().t()
        if torch.any((y - ref).abs() > w.shape[1] * 2.0 ** -23 * bound + 1e-30):
            raise RuntimeError(f"MXFP4 fused GEMM tensor {t} outside the fp32 summation bound")
    setup_s = time.perf_counter() - t0

    flat = wc.encode([("fp4_e2m1", np.ascontiguousarray(t.data).reshape(-1)) for t in blocks],
                     lanes=64, threads=args.threads)
    dflat = wc.to_device(flat, dev)
    outs = [torch.empty(n, dtype=torch.uint8, device=dev) for n in flat.out_bytes]

    # every variant rotates over resident copies of its weights (>= 1 GiB): the
    # fused one over copies of the blob and the scales
    sbytes = sum(s.numel() for s in dsc)
    n_f = rotation_copies(blob.size + sbytes)
    fcop = [(dblob, dsc)] + [(dblob.clone(), [s.clone() for s in dsc]) for _ in range(n_f - 1)]
    n_u = rotation_copies(flat.size + sum(flat.out_bytes) + sbytes)
    ucop = [(dflat, outs, dsc)] + [(dflat.clone(), [torch.empty_like(o) for o in outs],
                                    [s.clone() for s in dsc]) for _ in range(n_u - 1)]
    n_p = rotation_copies(sum(w.numel() * 2 for w in Wb))
    Wbs = [Wb] + [[w.clone() for w in Wb] for _ in range(n_p - 1)]

    def fused_k(k):
        d, sc = fcop[k % n_f]
        wc.gemv_mx(blob, d.data_ptr(), list(range(len(blocks))), [s.data_ptr() for s in sc],
                   [x.data_ptr() for x in xs], M, [y.data_ptr() for y in ys],
                   stream.cuda_stream, err.data_ptr())

    def unfused(k):
        d, o_k, sc = ucop[k % n_u]
        wc.decode(flat, d.data_ptr(), [o.data_ptr() for o in o_k], stream.cuda_stream,
                  err.data_ptr())
        for o, s, x, shp in zip(o_k, sc, xs, shapes):
            torch.matmul(x, dequant(o, s, shp).t())

    def uncompressed(k):
        for w, x in zip(Wbs[k % n_p], xs):
            torch.matmul(x, w.t())

    s_fused, s_unfused, s_plain = (timed_rotating(f, args.warmup, args.steps, stream)
                                   for f in (fused_k, unfused, uncompressed))
    read_gbps = hbm_read_rate(dev, stream)
    if int(err.item()):
        raise RuntimeError(f"device errors: {wc.describe_errors(int(err.item()))}")
    wbytes = sum(blob.out_bytes)
    alg = (blob.size + sbytes + sum(x.numel() * 2 for x in xs) +
           sum(2 * y.numel() * 4 for y in ys))
    achieved = alg / s_fused / 1e9
    line = {
        "metric": METRIC + " [fused MXFP4 decode-GEMM]",
        "value": round(wbytes / s_fused / 1e9, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(s_fused * 1e3, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "fp4 e2m1 x e8m0 (as bf16) x bf16 -> fp32",
        "data": "synthetic",
        "config": {"workload": workload, "mode": "fused-gemv-mx", "m": M,
                   "tile": f"{tile[0]}x{tile[1]} codes", "tile_order": "column-blocks",
                   "symbols": "bytes (two codes)" if args.mx_bytes else "e2m1 nibbles",
                   "product": "v_cvt_scalef32_pk_bf16_fp4 + v_mfma_f32_16x16x32_bf16",
                   "lanes": 64, "code_bytes_per_step": wbytes, "scale_bytes_per_step": sbytes,
                   "compressed_bytes_per_step": blob.size,
                   "copies_resident": {"fused": n_f, "unfused": n_u, "uncompressed": n_p},
                   "parallelism": "single-gpu"},
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBPS, 4), "traffic": None,
                     "kernel": gemv_kernel_for("mxfp4-bytes" if args.mx_bytes else "mxfp4",
                                               blob.n_chunks, M),
                     "mean_step_us": round(s_fused * 1e6, 2),
                     "algorithmic_bytes_per_step": int(alg)},
        "unfused": {"value": round(wbytes / s_unfused / 1e9, 2), "unit": "GB/s",
                    "ms_per_step": round(s_unfused * 1e3, 4),
                    "what": "wc_decode of the codes (64 KiB byte-run chunks), torch dequantisation "
                            "to bf16 with the scales, torch.matmul per tensor"},
        "uncompressed": {"value": round(wbytes / s_plain / 1e9, 2), "unit": "GB/s",
                         "ms_per_step": round(s_plain * 1e3, 4),
                         "what": "torch.matmul on the weights kept resident as bf16 (4x the "
                                 "fp4 bytes)"},
        "raw_codes_read": {"bytes": wbytes + sbytes,
                           "ms": round((wbytes + sbytes) / read_gbps / 1e6, 4),
                           "read_GBps": round(read_gbps, 1),
                           "what": "the uncompressed format's floor: its packed e2m1 codes and "
                                   "scales read once at the rate wc_stream reads 1 GiB"},
        "setup_s": round(setup_s, 1),
    }
    print(json.dumps(line), flush=True)
    return 0


def gemv_w4_bench(args, dev) -> int:
    """Fused decode-GEMM over the seven int4 projections of the 8B AWQ-style layer
    (or the symmetric int4 layer): codes as the blob's bytes, fp16 scales and
    zero points decoded once, bf16 x, fp32 y; checked against torch's fp32
    product of the same values."""
    import numpy as np
    import torch

    from paper_2606_15789_amd import synth, wc
    M = args.gemv_w4
    if not 1 <= M <= 64:
        print("--gemv-w4 takes 1..64 rows of activations", file=sys.stderr)
        return 2
    workload = "llama3-8b-layer-int4" if args.w4_signed else "llama3-8b-layer-awq4"
    tile = (16, 1024)   # bytes: 2048 codes
    t0 = time.perf_counter()
    ts = synth.config(WORKLOADS[workload])
    codes = [t for t in ts if t.name.endswith(".qweight")]
    scales = [t for t in ts if t.name.endswith(".scales")]
    zeros = [t for t in ts if t.name.endswith(".qzeros")]
    shapes = [t.shape for t in codes]
    if args.w4_nibbles:
        blob = wc.encode([("u4", t.data, t.shape) for t in codes], lanes=64,
                         tile=(tile[0], 2 * tile[1]), tile_order=1, threads=args.threads)
    else:
        blob = wc.encode([("u8", t.data, (t.shape[0], t.shape[1] // 2)) for t in codes],
                         lanes=64, tile=tile, tile_order=1, threads=args.threads)
    dblob = wc.to_device(blob, dev)
    dsc = [torch.from_numpy(np.ascontiguousarray(s.data).reshape(-1).view(np.int16)).to(dev)
           for s in scales]
    dz = None
    if zeros:
        dz = []
        for z in zeros:
            zp = torch.from_numpy(np.ascontiguousarray(z.data).reshape(-1)).to(dev)
            dz.append(torch.stack([zp & 15, zp >> 4], dim=1).reshape(-1).contiguous())

    def dequant(packed, j, shp):
        """bf16 weights s (q - z) or s q of packed codes (as exact as bf16 allows)."""
        p = packed.view(shp[0], shp[1] // 2)
        q = torch.stack([p & 15, p >> 4], dim=2).reshape(shp).int()
        if dz is None:
            q = (q ^ 8) - 8
        else:
            q = q - dz[j].view(shp[0], shp[1] // 128).int().repeat_interleave(128, dim=1)
        s = dsc[j].view(torch.float16).float().view(shp[0], shp[1] // 128)
        return (q.float() * s.repeat_interleave(128, dim=1)).to(torch.bfloat16)

    Wb = [dequant(torch.from_numpy(np.ascontiguousarray(t.data).reshape(-1)).to(dev), j, shp)
          for j, (t, shp) in enumerate(zip(codes, shapes))]
    gen = torch.Generator(device=dev)
    gen.manual_seed(24601)
    xs = [torch.randn(M, shp[1], generator=gen, device=dev).to(torch.bfloat16) for shp in shapes]
    ys = [torch.zeros(M, shp[0], dtype=torch.float32, device=dev) for shp in shapes]
    err = torch.zeros(1, dtype=torch.int32, device=dev)
    stream = torch.cuda.current_stream(dev)

    def fused():
        wc.gemv_w4(blob, dblob.data_ptr(), list(range(len(codes))), [s.data_ptr() for s in dsc],
                   None if dz is None else [z.data_ptr() for z in dz],
                   [x.data_ptr() for x in xs], M, [y.data_ptr() for y in ys],
                   stream.cuda_stream, err.data_ptr())

    fused()
    torch.cuda.synchronize()
    if int(err.item()):
        raise RuntimeError(f"device errors: {wc.describe_errors(int(err.item()))}")
    for t, (x, y, shp) in enumerate(zip(xs, ys, shapes)):
        # reference in fp32 from the exact weights s (q - z) (the bf16 copy rounds them)
        p = torch.from_numpy(np.ascontiguousarray(codes[t].data).reshape(-1)).to(dev)
        p = p.view(shp[0], shp[1] // 2)
        q = torch.stack([p & 15, p >> 4], dim=2).reshape(shp).int()
        q = (q ^ 8) - 8 if dz is None else \
            q - dz[t].view(shp[0], shp[1] // 128).int().repeat_interleave(128, dim=1)
        sg = dsc[t].view(torch.float16).double().view(shp[0], shp[1] // 128)
        s = sg.repeat_interleave(128, 1)
        w = q.double() * s
        xd = x.double()
        ref = xd @ w.t()
        # the derived fp32 bound of the fused product (group sums of x (16 + t) and
        # of x, the zero-point correction, the scale, the accumulation over groups
        # and tiles): u (10^4 sum_g |s_g| sum_{k in g} |x_k| + (K/128 + 64) sum |x w|)
        gx = xd.abs().view(x.shape[0], shp[1] // 128, 128).sum(dim=2)
        bound = 2.0 ** -24 * (1e4 * (gx @ sg.abs().t())
                              + (shp[1] / 128 + 64) * (xd.abs() @ w.abs().t()))
        if torch.any((y.double() - ref).abs() > bound + 1e-30):
            raise RuntimeError(f"int4 fused GEMM tensor {t} outside the fp32 error bound")
        del w, ref
    setup_s = time.perf_counter() - t0

    flat = wc.encode([("u8", np.ascontiguousarray(t.data).reshape(-1)) for t in codes],
                     lanes=64, threads=args.threads)
    dflat = wc.to_device(flat, dev)
    outs = [torch.empty(n, dtype=torch.uint8, device=dev) for n in flat.out_bytes]

    # every variant rotates over resident copies of its weights (>= 1 GiB): the
    # fused one over copies of the blob, the scales and the zero points
    aux = sum(s.numel() * 2 for s in dsc) + (sum(z.numel() for z in dz) if dz else 0)
    n_f = rotation_copies(blob.size + aux)
    fcop = [(dblob, dsc, dz)] + [(dblob.clone(), [s.clone() for s in dsc],
                                  None if dz is None else [z.clone() for z in dz])
                                 for _ in range(n_f - 1)]
    n_u = rotation_copies(flat.size + sum(flat.out_bytes) + aux)
    ucop = [(dflat, outs)] + [(dflat.clone(), [torch.empty_like(o) for o in outs])
                              for _ in range(n_u - 1)]
    n_p = rotation_copies(sum(w.numel() * 2 for w in Wb))
    Wbs = [Wb] + [[w.clone() for w in Wb] for _ in range(n_p - 1)]

    def fused_k(k):
        d, sc, zp = fcop[k % n_f]
        wc.gemv_w4(blob, d.data_ptr(), list(range(len(codes))), [s.data_ptr() for s in sc],
                   None if zp is None else [z.data_ptr() for z in zp],
                   [x.data_ptr() for x in xs], M, [y.data_ptr() for y in ys],
                   stream.cuda_stream, err.data_ptr())

    def unfused(k):
        d, o_k = ucop[k % n_u]
        wc.decode(flat, d.data_ptr(), [o.data_ptr() for o in o_k], stream.cuda_stream,
                  err.data_ptr())
        for j, (o, x, shp) in enumerate(zip(o_k, xs, shapes)):
            torch.matmul(x, dequant(o, j, shp).t())

    def uncompressed(k):
        for w, x in zip(Wbs[k % n_p], xs):
            torch.matmul(x, w.t())

    s_fused, s_unfused, s_plain = (timed_rotating(f, args.warmup, args.steps, stream)
                                   for f in (fused_k, unfused, uncompressed))
    read_gbps = hbm_read_rate(dev, stream)
    if int(err.item()):
        raise RuntimeError(f"device errors: {wc.describe_errors(int(err.item()))}")
    wbytes = sum(blob.out_bytes)
    alg = blob.size + aux + sum(x.numel() * 2 for x in xs) + sum(2 * y.numel() * 4 for y in ys)
    achieved = alg / s_fused / 1e9
    line = {
        "metric": METRIC + " [fused int4 decode-GEMM]",
        "value": round(wbytes / s_fused / 1e9, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(s_fused * 1e3, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int4 x fp16 scale (as bf16 16 + t) x bf16 -> fp32",
        "data": "synthetic",
        "config": {"workload": workload, "mode": "fused-gemv-w4", "m": M,
                   "tile": f"{tile[0]}x{2 * tile[1]} codes", "tile_order": "column-blocks",
                   "symbols": "nibbles" if args.w4_nibbles else "bytes (two codes)",
                   "zero_points": dz is not None,
                   "product": "v_perm + v_lshl_or to bf16 + v_mfma_f32_16x16x32_bf16 (x and ones)",
                   "lanes": 64, "code_bytes_per_step": wbytes, "aux_bytes_per_step": aux,
                   "compressed_bytes_per_step": blob.size,
                   "copies_resident": {"fused": n_f, "unfused": n_u, "uncompressed": n_p},
                   "parallelism": "single-gpu"},
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBPS, 4), "traffic": None,
                     "kernel": gemv_kernel_for("int4" if args.w4_nibbles else "int4-bytes",
                                               blob.n_chunks, M),
                     "mean_step_us": round(s_fused * 1e6, 2),
                     "algorithmic_bytes_per_step": int(alg)},
        "unfused": {"value": round(wbytes / s_unfused / 1e9, 2), "unit": "GB/s",
                    "ms_per_step": round(s_unfused * 1e3, 4),
                    "what": "wc_decode of the codes (64 KiB byte-run chunks), torch dequantisation "
                            "to bf16 with scales and zero points, torch.matmul per tensor"},
        "uncompressed": {"value": round(wbytes / s_plain / 1e9, 2), "unit": "GB/s",
                         "ms_per_step": round(s_plain * 1e3, 4),
                         "what": "torch.matmul on the dequantised weights kept resident as bf16 "
                                 "(4x the int4 bytes)"},
        "raw_codes_read": {"bytes": wbytes + aux,
                           "ms": round((wbytes + aux) / read_gbps / 1e6, 4),
                           "read_GBps": round(read_gbps, 1),
                           "what": "the uncompressed format's floor: its packed int4 codes, "
                                   "scales and zero points read once at the rate wc_stream "
                                   "reads 1 GiB"},
        "setup_s": round(setup_s, 1),
    }
    print(json.dumps(line), flush=True)
    return 0


def encode_bench(args, dev) -> int:
    """Device encoder (histograms, tables, chunk encode, index, packing) over
    one resident 70B layer: a step is one wc_encode_device call."""
    import numpy as np
    import torch

    import oracle
    from paper_2606_15789_amd import synth, wc
    t0 = time.perf_counter()
    tens = synth.config_torch_device(5, 0, device="cuda")
    entries = [("bf16", t, shape) for _, t, shape in tens]
    kw = dict(chunk_bytes=args.chunk_bytes, lanes=args.lanes)
    cap, wsb = wc.encode_device_bounds(entries, **kw)
    blob = torch.empty(cap, dtype=torch.uint8, device=dev)
    ws = torch.empty(wsb, dtype=torch.uint8, device=dev)
    size = torch.zeros(1, dtype=torch.int64, device=dev)
    stream = torch.cuda.current_stream(dev)

    def step():
        wc.encode_device(entries, blob=blob, workspace=ws, size=size, stream=stream, **kw)

    # correctness: the device blob is the host encoder's blob, and it decodes
    step()
    torch.cuda.synchronize()
    n = int(size.item())
    got = blob[:n].cpu().numpy()
    host = [(dt, t.cpu().numpy(), shape) for dt, t, shape in entries]
    h0 = time.perf_counter()
    ref = wc.encode(host, threads=args.threads, **kw)
    host_s = time.perf_counter() - h0
    if n != ref.size or not np.array_equal(got, ref.array()):
        raise RuntimeError("device blob differs from the host encoder's")
    err = torch.zeros(1, dtype=torch.int32, device=dev)
    outs = wc.decode_torch(ref, blob, err=err)
    torch.cuda.synchronize()
    if int(err.item()) or any(not torch.equal(o, t) for o, (_, t, _) in zip(outs, entries)):
        raise RuntimeError("device blob does not decode to the layer")
    del outs, got
    out_bytes = sum(ref.out_bytes)
    setup_s = time.perf_counter() - t0

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    K = args.steps
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(K)]
    for k in range(K):
        ev[k][0].record(stream)
        step()
        ev[k][1].record(stream)
    torch.cuda.synchronize()
    ms = [a.elapsed_time(b) for a, b in ev]
    if int(size.item()) != n:
        raise RuntimeError("timed encodes gave another size")
    mean_s = float(np.mean(ms)) / 1e3
    alg = out_bytes + n  # the layer read once, the blob written once
    cpu = None
    if not args.no_cpu_baseline:
        # oracle encode of the k and v projections on one core
        sample = [(dt, h, shape) for dt, h, shape in host if shape[0] == 1024]
        old = os.sched_getaffinity(0)
        core = min(old)
        os.sched_setaffinity(0, {core})
        reps, dt = 0, 0.0
        try:
            while reps == 0 or dt < 3.0:
                c0 = time.perf_counter()
                ob = oracle.encode(sample, **kw)
                dt += time.perf_counter() - c0
                reps += 1
        finally:
            os.sched_setaffinity(0, old)
        if ob != wc.encode(sample, threads=args.threads, **kw).tobytes():
            raise RuntimeError("oracle sample blob differs")
        sb = sum(h.nbytes for _, h, _ in sample)
        cpu = {"value": round(reps * sb / dt / 1e9, 4), "unit": "GB/s", "cores": 1,
               "kind": "oracle",
               "sample": f"oracle encode of the k_proj and v_proj tensors ({sb} bytes) of the "
                         f"70B layer, {reps}x, single thread pinned to core {core}",
               "seconds": round(dt, 3), "cpu": cpu_model(), "host_cpus": os.cpu_count()}
    line = {
        "metric": "encoded GB/s of weights on one MI355X (% of HBM roofline)",
        "value": round(out_bytes / mean_s / 1e9, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": round(mean_s * 1e3, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u32",
        "data": "synthetic",
        "config": {"workload": "llama3-70b-layer-bf16", "mode": "device-encode",
                   "input_bytes_per_step": out_bytes, "blob_bytes_per_step": n,
                   "chunk_bytes": args.chunk_bytes, "lanes": args.lanes,
                   "parallelism": "single-gpu"},
        "roofline": {"bound": "hbm", "achieved": round(alg / mean_s / 1e9, 1),
                     "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": round(alg / mean_s / 1e9 / HBM_PEAK_GBPS, 4), "traffic": None,
                     "kernel": "wc_encode_device (7 launches)",
                     "mean_step_us": round(mean_s * 1e6, 2),
                     "algorithmic_bytes_per_step": int(alg)},
        "cpu_baseline": cpu,
        "host_library_encode": {"value": round(out_bytes / host_s / 1e9, 3), "unit": "GB/s",
                                "threads": args.threads, "seconds": round(host_s, 3)},
        "setup_s": round(setup_s, 1),
    }
    print(json.dumps(line), flush=True)
    return 0


def sweep_bench(args, dev) -> int:
    """Decode throughput and compression of one bf16 decoder layer per model
    family (qwen2-1.5b .. llama3-405b).  Each layer is drawn on the GPU,
    compressed by wc_encode_device, checked to decode back bit-exact, and
    decoded K times from resident blobs (copies rotated so at least 1 GiB of
    blobs and outputs is touched, as for the other small workloads)."""
    import numpy as np
    import torch

    from paper_2606_15789_amd import synth, wc
    stream = torch.cuda.current_stream(dev)
    err = torch.zeros(1, dtype=torch.int32, device=dev)
    ws = torch.empty(wc.ANALYZE_WORKSPACE_BYTES, dtype=torch.uint8, device=dev)
    for seed, (model, (shapes, sigma)) in enumerate(synth.MODEL_LAYERS.items(), start=20):
        t0 = time.perf_counter()
        tens = synth.layer_torch_device(shapes, sigma, seed, device="cuda")
        entries = [("bf16", t, shape) for _, t, shape in tens]
        kw = dict(chunk_bytes=args.chunk_bytes, lanes=args.lanes)
        dblob, size = wc.encode_device(entries, **kw)
        torch.cuda.synchronize()
        n = int(size.item())
        dblob = dblob[:n].clone()
        blob = wc.open_blob(dblob.cpu().numpy())
        stats = [wc.analyze_device("bf16", t, workspace=ws) for _, t, _ in entries]
        bound = sum(st["bound_bytes"] for st in stats)
        out_b = sum(blob.out_bytes)
        n_res = max(1, -(-ROTATE_BYTES // (n + out_b)))
        dblobs = [dblob] + [dblob.clone() for _ in range(n_res - 1)]
        outs = [[torch.empty(b, dtype=torch.uint8, device=dev) for b in blob.out_bytes]
                for _ in range(n_res)]
        for r in range(n_res):
            wc.decode_torch(blob, dblobs[r], outs=outs[r], err=err)
        torch.cuda.synchronize()
        if int(err.item()) or any(not torch.equal(o, t) for r in range(n_res)
                                  for o, (_, t, _) in zip(outs[r], entries)):
            raise RuntimeError(f"{model}: decode differs from the original layer")
        setup_s = time.perf_counter() - t0

        def step(k):
            r = k % n_res
            wc.decode(blob, dblobs[r].data_ptr(), [o.data_ptr() for o in outs[r]],
                      stream.cuda_stream, err.data_ptr())

        for k in range(args.warmup):
            step(k)
        torch.cuda.synchronize()
        K = args.steps
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
              for _ in range(K)]
        start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        start.record(stream)
        for k in range(K):
            ev[k][0].record(stream)
            step(args.warmup + k)
            ev[k][1].record(stream)
        end.record(stream)
        torch.cuda.synchronize()
        if int(err.item()):
            raise RuntimeError(f"{model}: device errors {wc.describe_errors(int(err.item()))}")
        last = (args.warmup + K - 1) % n_res
        if any(not torch.equal(o, t) for o, (_, t, _) in zip(outs[last], entries)):
            raise RuntimeError(f"{model}: timed decode differs from the original layer")
        total_ms = start.elapsed_time(end)
        mean_s = float(np.mean([a.elapsed_time(b) for a, b in ev])) / 1e3
        achieved = (n + out_b) / mean_s / 1e9
        line = {
            "metric": METRIC,
            "value": round(K * out_b / (total_ms / 1e3) / 1e9, 2),
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
            "config": {"workload": f"{model}-layer-bf16", "mode": "model-sweep",
                       "tensors_per_step": len(entries), "params": out_b // 2,
                       "decoded_bytes_per_step": out_b, "compressed_bytes_per_step": n,
                       "sigma": sigma, "chunk_bytes": args.chunk_bytes, "lanes": args.lanes,
                       "copies_resident": n_res, "parallelism": "single-gpu"},
            "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS,
                         "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBPS, 4),
                         "traffic": None,
                         "kernel": decode_kernel_for(["bf16"] * len(entries), blob.n_chunks,
                                                     args.lanes, False),
                         "mean_launch_us": round(mean_s * 1e6, 2),
                         "algorithmic_bytes_per_launch": int(n + out_b)},
            "compression": {"ratio": round(out_b / n, 5), "bound_ratio": round(out_b / bound, 5),
                            "payload_over_bound_pct":
                                round(100 * (blob.payload_bytes() / bound - 1), 4),
                            "total_over_bound_pct": round(100 * (n / bound - 1), 4)},
            "cpu_baseline": None,
            "setup_s": round(setup_s, 1),
        }
        print(json.dumps(line), flush=True)
        del tens, entries, dblob, dblobs, outs, blob
        torch.cuda.empty_cache()
    return 0


if __name__ == "__main__":
    sys.exit(main())
