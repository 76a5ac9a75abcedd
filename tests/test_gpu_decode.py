"""GPU parity: libwc's HIP decode against the oracle and the original bytes.

Every case decodes through the C ABI (wc_decode) on cuda:0 and requires the
output to be bit-identical to the original tensor and to the oracle's decode
of the same blob (whole blob at small sizes; sampled chunks, decoded one by
one by the oracle, at the full workload sizes).
"""
import os
import struct
import sys

import numpy as np
import pytest

import oracle
from paper_2606_15789_amd import synth, wc

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda:0")


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def gpu_decode(blob, dev, expect_err=0):
    dblob = wc.to_device(blob, dev)
    err = torch.zeros(1, dtype=torch.int32, device=dev)
    outs = wc.decode_torch(blob, dblob, err=err)
    torch.cuda.synchronize()
    assert int(err.item()) == expect_err, wc.describe_errors(int(err.item()))
    return outs


def check_exact(pairs, blob, outs, oracle_full=True):
    ref = oracle.decode(blob.tobytes()) if oracle_full else None
    for t, ((dt, data), out) in enumerate(zip(pairs, outs)):
        got = out.cpu().numpy()
        orig = np.ascontiguousarray(data).view(np.uint8).reshape(-1)
        assert np.array_equal(got, orig), (t, dt)
        if ref is not None:
            assert np.array_equal(got, ref[t]), (t, dt)


@pytest.mark.parametrize("lanes", [64, 32])
def test_every_bit_pattern(dev, lanes):
    rng = np.random.default_rng(0)
    allw = rng.permutation(np.arange(65536, dtype=np.uint32)).astype(np.uint16)
    pairs = [("bf16", allw), ("fp16", allw[::-1].copy()),
             ("u8", rng.permutation(np.repeat(np.arange(256, dtype=np.uint8), 40))),
             ("u4", rng.permutation(np.repeat(np.arange(256, dtype=np.uint8), 40))),
             ("fp8_e4m3", rng.permutation(np.repeat(np.arange(256, dtype=np.uint8), 30))),
             ("fp8_e5m2", rng.permutation(np.repeat(np.arange(256, dtype=np.uint8), 20))),
             ("fp4_e2m1", rng.permutation(np.repeat(np.arange(256, dtype=np.uint8), 25)))]
    for cb in (256, 16384, 65536):
        say("bit patterns, chunk", cb, "lanes", lanes)
        blob = wc.encode(pairs, chunk_bytes=cb, lanes=lanes)
        check_exact(pairs, blob, gpu_decode(blob, dev))


@pytest.mark.parametrize("dtype,esize", [("bf16", 2), ("fp16", 2), ("u8", 1), ("u4", 1),
                                         ("fp8_e4m3", 1), ("fp4_e2m1", 1)])
@pytest.mark.parametrize("cb", [256, 16384, 65536])
@pytest.mark.parametrize("lanes", [64, 32])
def test_edge_sizes(dev, dtype, esize, cb, lanes):
    rng = np.random.default_rng(1)
    E = cb // esize
    sizes = [0, 1, 2, 3, 5, 63, 64, 65, 127, 128, 129, 255, 257, E - 1, E, E + 1, 2 * E + 7, 3 * E]
    pairs = []
    for n in sizes:
        if esize == 2:
            d = (rng.normal(0, 0.02, n).astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
        else:
            d = rng.integers(0, 256, n).astype(np.uint8)
            d[: n // 2] = 3
        pairs.append((dtype, d))
    say("edge sizes", dtype, cb, "lanes", lanes)
    blob = wc.encode(pairs, chunk_bytes=cb, lanes=lanes)
    check_exact(pairs, blob, gpu_decode(blob, dev))


@pytest.mark.parametrize("lanes", [64, 32])
def test_degenerate_tables(dev, lanes):
    pairs = [("u8", np.full(200_000, 42, np.uint8)),                 # single symbol: f = 4096
             ("u4", np.full(70_000, 0x77, np.uint8)),
             ("bf16", np.full(50_000, 0x3F80, np.uint16)),
             ("u8", np.concatenate([np.zeros(100_000, np.uint8), np.arange(256, dtype=np.uint8)])),
             ("u8", np.arange(256, dtype=np.uint8).repeat(300))]     # uniform: 8 bits
    blob = wc.encode(pairs, lanes=lanes)
    check_exact(pairs, blob, gpu_decode(blob, dev))


@pytest.mark.parametrize("cfg,div", [(1, 4), (2, 8), (3, 8), (4, 8), (5, 16), (6, 8), (7, 8),
                                     (8, 8), (9, 8)])
@pytest.mark.parametrize("lanes", [64, 32])
def test_workloads_scaled(dev, cfg, div, lanes):
    say("workload", cfg, "div", div, "lanes", lanes)
    pairs = [(t.dtype, t.data) for t in synth.config(cfg, div=div)]
    blob = wc.encode(pairs, lanes=lanes)
    check_exact(pairs, blob, gpu_decode(blob, dev))


@pytest.mark.parametrize("cfg", [3, 7, 8])
def test_nibble_tensors_coded_by_bytes(dev, cfg):
    """4-bit tensors (int4, MXFP4, AWQ-style codes) coded by their packed bytes,
    two nibbles per symbol: the host blob equals the oracle's and the GPU decode
    is bit-exact."""
    say("nibbles as bytes", cfg)
    pairs = [("u8" if t.dtype in ("u4", "fp4_e2m1") else t.dtype, t.data)
             for t in synth.config(cfg, div=8)]
    blob = wc.encode(pairs)
    assert blob.tobytes() == oracle.encode(pairs)
    check_exact(pairs, blob, gpu_decode(blob, dev))


def test_oracle_blob_decodes_on_gpu(dev):
    pairs = [(t.dtype, t.data) for t in synth.config(3, div=8)]
    blob = wc.open_blob(oracle.encode(pairs, chunk_bytes=32768))
    check_exact(pairs, blob, gpu_decode(blob, dev), oracle_full=False)


@pytest.mark.parametrize("lanes", [64, 32])
def test_many_tensors_split_over_launches(dev, lanes):
    rng = np.random.default_rng(4)
    pairs = []
    for i in range(75):
        dt = ["bf16", "u8", "u4", "fp16"][i % 4]
        n = int(rng.integers(0, 70_000))
        if dt in ("bf16", "fp16"):
            d = (rng.normal(0, 0.05, n).astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
        else:
            d = rng.integers(0, 40, n).astype(np.uint8)
        pairs.append((dt, d))
    blob = wc.encode(pairs, chunk_bytes=16384, lanes=lanes)
    check_exact(pairs, blob, gpu_decode(blob, dev))


def _sample_chunks(n, k, rng):
    if n <= k:
        return list(range(n))
    pick = set([0, n - 1]) | set(int(c) for c in rng.choice(n, size=k - 2, replace=False))
    return sorted(pick)


@pytest.mark.parametrize("cfg,lanes", [(1, 64), (2, 64), (3, 64), (4, 64), (5, 64), (4, 32),
                                       (5, 32), (6, 64), (7, 64), (8, 64), (9, 64)])
def test_workloads_full_size(dev, cfg, lanes):
    """Full workload sizes in the benchmark's launch configuration (one launch)."""
    say("full workload", cfg, "lanes", lanes)
    ts = synth.config(cfg)
    pairs = [(t.dtype, t.data) for t in ts]
    blob = wc.encode(pairs, chunk_bytes=65536, lanes=lanes)
    outs = gpu_decode(blob, dev)
    rng = np.random.default_rng(cfg)
    raw = blob.tobytes()
    info = oracle.tensor_info(raw)
    for t, ((dt, data), out) in enumerate(zip(pairs, outs)):
        orig = torch.from_numpy(np.ascontiguousarray(data).view(np.uint8).reshape(-1)).to(dev)
        assert torch.equal(out, orig), (cfg, t)
        got = out.cpu().numpy()
        for c in _sample_chunks(info[t]["n_chunks"], 12, rng):
            ref = oracle.decode_chunks(raw, t, c, c + 1)
            lo, hi = c * 65536, min((c + 1) * 65536, info[t]["out_bytes"])
            assert np.array_equal(got[lo:hi], ref[lo:hi]), (cfg, t, c)
    del outs
    torch.cuda.empty_cache()


@pytest.mark.parametrize("rows,cols,dtype", [(6144, 32768, "bf16"), (6145, 32768, "bf16"),
                                             (7000, 32704, "bf16"), (7000, 32704, "fp16"),
                                             (8192, 32768, "bf16"), (8193, 32768, "bf16")])
def test_launches_around_the_wide_kernels_window(dev, rows, cols, dtype):
    """wc_decode runs a bf16 launch of untiled 64-lane chunks on its 16-wave
    kernel when the chunks overflow the general kernel's resident waves (6144
    on a 256-CU MI355X) but fit in the 16-wave kernel's (8192).  Chunk counts
    on both edges of that window (the 7000-row case ends in a partial chunk)
    decode bit-exact; sampled chunks equal the oracle's decode; a flipped word
    in the wide launch is reported like in the general one.  The fp16 case
    codes the same 16-bit words as fp16 (the split is the same bit fields)."""
    say("wide window", rows, cols, dtype)
    (_, t, shape), = synth.layer_torch_device([("w", rows, cols)], 0.02, 40 + rows % 97)
    blob, size = wc.encode_device([(dtype, t, shape)])
    torch.cuda.synchronize()
    raw = blob[:int(size.item())].cpu().numpy()
    desc = wc.open_blob(raw)
    rawb = raw.tobytes()
    info = oracle.tensor_info(rawb)
    say(f"  {info[0]['n_chunks']} chunks, {t.numel() / 1e9:.3f} GB")
    err = torch.zeros(1, dtype=torch.int32, device=dev)
    out, = wc.decode_torch(desc, blob, err=err)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    assert torch.equal(out, t)
    got = out.cpu().numpy()
    rng = np.random.default_rng(rows)
    for c in _sample_chunks(info[0]["n_chunks"], 6, rng):
        ref = oracle.decode_chunks(rawb, 0, c, c + 1)
        lo, hi = c * 65536, min((c + 1) * 65536, info[0]["out_bytes"])
        assert np.array_equal(got[lo:hi], ref[lo:hi]), c
    del out
    # a flipped word in the middle chunk's record
    c = info[0]["n_chunks"] // 2
    idx = struct.unpack_from("<Q", rawb, 32)[0]
    off = struct.unpack_from("<I", rawb, idx + 4 * c)[0] * 16
    nw, na = struct.unpack_from("<II", rawb, off)
    wpos = off + 16 + ((4 * na + 15) // 16) * 16 + 2 * (nw // 2)
    blob[wpos] ^= 0x40
    err.zero_()
    wc.decode_torch(desc, blob, err=err)
    torch.cuda.synchronize()
    assert int(err.item()) & 0x6
    del blob, t
    torch.cuda.empty_cache()


@pytest.mark.parametrize("lanes", [64, 32])
def test_device_side_corruption_flags(dev, lanes):
    """The kernel's own checks turn corrupted device bytes into error bits."""
    pairs = [(t.dtype, t.data) for t in synth.config(1, div=8)]
    blob = wc.encode(pairs, chunk_bytes=16384, lanes=lanes)
    raw = blob.tobytes()
    idx = struct.unpack_from("<Q", raw, 32)[0]
    off1 = struct.unpack_from("<I", raw, idx + 4)[0] * 16
    nw, A = struct.unpack_from("<II", raw, off1)
    wpos = off1 + 16 + ((4 * A + 15) // 16) * 16 + 2 * (nw // 2)
    foff = struct.unpack_from("<Q", raw, 64 + 48)[0]

    def run(mutate):
        d = wc.to_device(blob, dev)
        mutate(d)
        err = torch.zeros(1, dtype=torch.int32, device=dev)
        wc.decode_torch(blob, d, err=err)
        torch.cuda.synchronize()
        return int(err.item())

    def flip_word(d):
        d[wpos] ^= 0x40

    def bump_state(d):
        d[off1 + 16 + 20] ^= 0x01

    def break_index(d):
        d[idx + 4: idx + 8] = 0

    def bad_header(d):
        d[off1: off1 + 4] = torch.tensor([0xFF, 0xFF, 0, 0], dtype=torch.uint8, device=dev)

    def bad_table(d):
        d[foff + 2] = (int(d[foff + 2].item()) + 1) & 0xFF

    assert run(lambda d: None) == 0
    assert run(flip_word) & 0x6
    assert run(bump_state) & 0x6
    assert run(break_index) & 0x1
    assert run(bad_header) & 0x1
    assert run(bad_table) & 0x8


def test_null_error_pointer_and_stream(dev):
    pairs = [(t.dtype, t.data) for t in synth.config(4, div=16)]
    blob = wc.encode(pairs)
    d = wc.to_device(blob, dev)
    s = torch.cuda.Stream(dev)
    with torch.cuda.stream(s):
        outs = wc.decode_torch(blob, d, stream=s)
    s.synchronize()
    check_exact(pairs, blob, outs, oracle_full=False)


def _shaped(ts):
    return [(t.dtype, t.data, t.shape if len(t.shape) == 2 else None) for t in ts]


@pytest.mark.parametrize("tile", [(32, 128), (64, 256), (128, 256), (1, 256)])
@pytest.mark.parametrize("lanes", [64, 32])
def test_tiled_workloads_scaled(dev, tile, lanes):
    """2-D tiles (one chunk per tile) with a layer codebook: every tensor the
    tile divides is written through the tile addressing, the rest stay flat."""
    say("tiles", tile, "lanes", lanes)
    ts = synth.config(2, div=8) + synth.config(3, div=8) + synth.config(7, div=8)
    pairs = _shaped(ts)
    blob = wc.encode(pairs, chunk_bytes=16384, lanes=lanes, tile=tile, codebook="layer")
    assert any(i["tile"] == tile for i in oracle.tensor_info(blob.tobytes()))
    check_exact([(d, a) for d, a, _ in pairs], blob, gpu_decode(blob, dev))


def test_tiled_full_size_70b_layer(dev):
    """The 70B layer in 128 x 256 tiles (64 KiB each) with one bf16 codebook."""
    ts = synth.config(5)
    pairs = _shaped(ts)
    blob = wc.encode(pairs, lanes=64, tile=(128, 256), codebook="layer")
    outs = gpu_decode(blob, dev)
    raw = blob.tobytes()
    info = oracle.tensor_info(raw)
    rng = np.random.default_rng(5)
    for t, ((dt, data, shape), out) in enumerate(zip(pairs, outs)):
        orig = torch.from_numpy(np.ascontiguousarray(data).view(np.uint8).reshape(-1)).to(dev)
        assert torch.equal(out, orig), t
        got = out.cpu().numpy().view(np.uint16).reshape(shape)
        ntc = shape[1] // 256
        for c in _sample_chunks(info[t]["n_chunks"], 6, rng):
            ref = oracle.decode_chunks(raw, t, c, c + 1).view(np.uint16).reshape(shape)
            a, b = divmod(c, ntc)
            rs, cs = slice(a * 128, (a + 1) * 128), slice(b * 256, (b + 1) * 256)
            assert np.array_equal(got[rs, cs], ref[rs, cs]), (t, c)
    del outs
    torch.cuda.empty_cache()
