"""GPU parity of the device-side analysis and encoder (wc_analyze_device,
wc_encode_device) against the oracle.

The device encoder must write the very blob the oracle's encoder writes from
the same tensors and parameters, byte for byte (the format fixes every
choice), so each case compares whole blobs: device == oracle, and == the host
library's wc_encode.  At full workload sizes the device blob is compared with
the host library's whole blob and decoded back on the GPU, and sampled chunks
are decoded one by one by the oracle.  The statistics must equal the oracle's
(integer histograms exactly, entropies to the last bit of the same formula).
"""
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


def to_dev(data, dev):
    b = np.ascontiguousarray(data).view(np.uint8).reshape(-1)
    return torch.from_numpy(b.copy()).to(dev)


def device_blob(entries, dev, **kw):
    """Device-encode host arrays; returns the blob bytes."""
    dents = [(e[0], to_dev(e[1], dev)) + tuple(e[2:]) for e in entries]
    blob, size = wc.encode_device(dents, **kw)
    torch.cuda.synchronize()
    n = int(size.item())
    cap, _ = wc.encode_device_bounds(dents, **kw)
    assert n <= cap == blob.numel()
    return blob[:n].cpu().numpy().tobytes()


def assert_same_blob(entries, dev, **kw):
    got = device_blob(entries, dev, **kw)
    want = oracle.encode([e[:2] + (e[2] if len(e) > 2 else None,) for e in entries], **kw)
    assert len(got) == len(want)
    if got != want:
        a, b = np.frombuffer(got, np.uint8), np.frombuffer(want, np.uint8)
        bad = np.flatnonzero(a != b)
        raise AssertionError(f"{bad.size} bytes differ, first at {bad[:8]}")
    host = wc.encode(entries, threads=4, **kw)
    assert host.tobytes() == got
    return got


def test_every_bit_pattern(dev):
    rng = np.random.default_rng(0)
    allw = rng.permutation(np.arange(65536, dtype=np.uint32)).astype(np.uint16)
    entries = [("bf16", allw), ("fp16", allw[::-1].copy()),
               ("u8", rng.permutation(np.repeat(np.arange(256, dtype=np.uint8), 40))),
               ("u4", rng.permutation(np.repeat(np.arange(256, dtype=np.uint8), 40))),
               ("fp8_e4m3", rng.permutation(np.repeat(np.arange(256, dtype=np.uint8), 30))),
               ("fp8_e5m2", rng.permutation(np.repeat(np.arange(256, dtype=np.uint8), 20))),
               ("fp4_e2m1", rng.permutation(np.repeat(np.arange(256, dtype=np.uint8), 25)))]
    for cb in (256, 16384, 65536):
        for lanes in (64, 32, 1, 7):
            say("bit patterns, chunk", cb, "lanes", lanes)
            assert_same_blob(entries, dev, chunk_bytes=cb, lanes=lanes)


@pytest.mark.parametrize("dtype,esize", [("bf16", 2), ("fp16", 2), ("u8", 1), ("u4", 1),
                                         ("fp8_e4m3", 1), ("fp4_e2m1", 1)])
@pytest.mark.parametrize("cb", [256, 16384, 65536])
def test_edge_sizes(dev, dtype, esize, cb):
    rng = np.random.default_rng(1)
    E = cb // esize
    sizes = [0, 1, 2, 3, 5, 63, 64, 65, 127, 128, 129, 255, 257, E - 1, E, E + 1, 2 * E + 7, 3 * E]
    entries = []
    for n in sizes:
        if esize == 2:
            d = (rng.normal(0, 0.02, n).astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
        else:
            d = rng.integers(0, 256, n).astype(np.uint8)
            d[: n // 2] = 3
        entries.append((dtype, d))
    for lanes in (64, 32):
        say("edge sizes", dtype, cb, "lanes", lanes)
        assert_same_blob(entries, dev, chunk_bytes=cb, lanes=lanes)


def test_degenerate_tables(dev):
    entries = [("u8", np.full(200_000, 42, np.uint8)),                 # f = 4096: no words
               ("u4", np.full(70_000, 0x77, np.uint8)),
               ("bf16", np.full(50_000, 0x3F80, np.uint16)),
               ("u8", np.concatenate([np.zeros(100_000, np.uint8), np.arange(256, dtype=np.uint8)])),
               ("u8", np.arange(256, dtype=np.uint8).repeat(300))]     # uniform: 8 bits
    for lanes in (64, 32):
        assert_same_blob(entries, dev, lanes=lanes)


def test_excess_normalisation(dev):
    """Many rare symbols force f = 1 and the excess comes off the largest f."""
    rng = np.random.default_rng(5)
    d = np.concatenate([np.zeros(4_000_000, np.uint8), np.arange(1, 256, dtype=np.uint8),
                        rng.integers(1, 256, 300).astype(np.uint8)])
    assert_same_blob([("u8", rng.permutation(d))], dev, chunk_bytes=16384)


@pytest.mark.parametrize("cfg,div", [(1, 4), (2, 8), (3, 8), (4, 8), (5, 16), (6, 8), (7, 8),
                                     (8, 8), (9, 8)])
def test_workloads_scaled(dev, cfg, div):
    say("workload", cfg, "div", div)
    entries = [(t.dtype, t.data) for t in synth.config(cfg, div=div)]
    for lanes in (64, 32):
        assert_same_blob(entries, dev, lanes=lanes)


def _shaped(ts):
    return [(t.dtype, t.data, t.shape if len(t.shape) == 2 else None) for t in ts]


@pytest.mark.parametrize("tile,order", [((32, 128), 0), ((64, 256), 0), ((128, 256), 0),
                                        ((1, 256), 0), ((64, 512), 1), ((32, 128), 1)])
@pytest.mark.parametrize("codebook", ["layer", "tensor"])
def test_tiles_and_codebooks(dev, tile, order, codebook):
    say("tiles", tile, "order", order, codebook)
    ts = synth.config(2, div=8) + synth.config(3, div=8) + synth.config(7, div=8)
    entries = _shaped(ts)
    for lanes in (64, 32):
        assert_same_blob(entries, dev, chunk_bytes=16384, lanes=lanes, tile=tile,
                         codebook=codebook, tile_order=order)


def test_many_tensors_over_launches(dev):
    rng = np.random.default_rng(4)
    entries = []
    for i in range(75):
        dt = ["bf16", "u8", "u4", "fp16"][i % 4]
        n = int(rng.integers(0, 70_000))
        if dt in ("bf16", "fp16"):
            d = (rng.normal(0, 0.05, n).astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
        else:
            d = rng.integers(0, 40, n).astype(np.uint8)
        entries.append((dt, d))
    assert_same_blob(entries, dev, chunk_bytes=16384)
    assert_same_blob(entries, dev, chunk_bytes=16384, codebook="layer")


def _sample_chunks(n, k, rng):
    if n <= k:
        return list(range(n))
    return sorted(set([0, n - 1]) | set(int(c) for c in rng.choice(n, size=k - 2, replace=False)))


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5])
def test_workloads_full_size(dev, cfg):
    """Full sizes: the device blob equals the host library's whole blob, decodes
    on the GPU to the original, and sampled chunks decode in the oracle."""
    say("full workload", cfg)
    ts = synth.config(cfg)
    entries = [(t.dtype, t.data) for t in ts]
    got = device_blob(entries, dev, chunk_bytes=65536, lanes=64)
    host = wc.encode(entries, chunk_bytes=65536, lanes=64)
    assert host.tobytes() == got
    del host
    blob = wc.open_blob(got)
    dblob = torch.from_numpy(np.frombuffer(got, np.uint8).copy()).to(dev)
    err = torch.zeros(1, dtype=torch.int32, device=dev)
    outs = wc.decode_torch(blob, dblob, err=err)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    rng = np.random.default_rng(cfg)
    info = oracle.tensor_info(got)
    for t, ((dt, data), out) in enumerate(zip(entries, outs)):
        orig = to_dev(data, dev)
        assert torch.equal(out, orig), (cfg, t)
        ob = np.ascontiguousarray(data).view(np.uint8).reshape(-1)
        for c in _sample_chunks(info[t]["n_chunks"], 8, rng):
            ref = oracle.decode_chunks(got, t, c, c + 1)
            lo, hi = c * 65536, min((c + 1) * 65536, info[t]["out_bytes"])
            assert np.array_equal(ob[lo:hi], ref[lo:hi]), (cfg, t, c)
    del outs, dblob
    torch.cuda.empty_cache()


def test_tensors_past_4_gib(dev):
    """The largest sizes: one blob of an int8 matrix of 65 541 x 65 533 symbols
    and a bf16 matrix of 131 073 x 16 384 (4 GiB + 32 KiB): symbol counts and
    output offsets pass 2^32, the bf16 chunk records straddle 4 GiB of blob and
    the raw region lies past it, and both tensors end in a partial chunk.  Encoded on the device,
    decoded on the GPU to the original bytes; sampled chunks (the first, the
    last, the two around 4 GiB of output, random ones) decoded by the oracle."""
    say("tensors past 4 GiB")
    i8 = synth.int8_rows_torch_device(65541, 65533, seed=11, device=dev)
    bf = synth.layer_torch_device([("w", 131073, 16384)], 0.02, 12, device=dev)[0][1]
    dents = [("u8", i8), ("bf16", bf)]
    blob, size = wc.encode_device(dents)
    torch.cuda.synchronize()
    n = int(size.item())
    host = blob[:n].cpu().numpy()
    desc = wc.open_blob(host)
    assert list(desc.out_bytes) == [65541 * 65533, 131073 * 32768]
    info = oracle.tensor_info(host)
    # header bytes 32 and 48: u64 offsets of the index (record offsets / 16)
    # and of the raw region, which sits between the index and the records; the
    # bf16 tensor's chunk records follow the int8 tensor's, all past 4 GiB
    index, raw = (int(host[o:o + 8].view(np.uint64)[0]) for o in (32, 48))
    g = info[0]["n_chunks"]
    first_bf16 = 16 * int(host[index + 4 * g:index + 4 * g + 4].view(np.uint32)[0])
    assert raw < 2**32 < first_bf16 < n, (raw, first_bf16, n)
    say("blob bytes", n, "bf16 records from", first_bf16, "raw region from", raw)
    err = torch.zeros(1, dtype=torch.int32, device=dev)
    outs = wc.decode_torch(desc, blob, err=err)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    for t, (x, out) in enumerate(zip((i8, bf), outs)):
        assert torch.equal(out, x), t
    del outs, blob
    torch.cuda.empty_cache()
    rng = np.random.default_rng(12)
    for t, x in enumerate((i8, bf)):
        ob, nc = info[t]["out_bytes"], info[t]["n_chunks"]
        c4 = 2**32 // 65536
        picks = sorted({0, nc - 1, c4 - 1, c4} | set(int(c) for c in rng.choice(nc, 6, False)))
        buf = np.zeros(ob, np.uint8)
        for c in picks:
            oracle.decode_chunks(host, t, c, c + 1, out=buf)
            lo, hi = c * 65536, min((c + 1) * 65536, ob)
            assert np.array_equal(buf[lo:hi], x[lo:hi].cpu().numpy()), (t, c)
    del i8, bf
    torch.cuda.empty_cache()


def test_round_trip_on_device_only(dev):
    """Encode and decode without the blob leaving the GPU (bar the descriptor)."""
    ts = synth.config(2, div=4)
    dents = [(t.dtype, to_dev(t.data, dev)) for t in ts]
    blob, size = wc.encode_device(dents, chunk_bytes=32768)
    torch.cuda.synchronize()
    n = int(size.item())
    desc = wc.open_blob(blob[:n].cpu().numpy())
    err = torch.zeros(1, dtype=torch.int32, device=dev)
    outs = wc.decode_torch(desc, blob, err=err)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    for (dt, x), out in zip(dents, outs):
        assert torch.equal(out, x)


def test_reused_buffers_and_stream(dev):
    """Two encodes into the same blob, workspace and size buffers on a side
    stream: the second (smaller) blob is whole and the bytes past it untouched."""
    rng = np.random.default_rng(9)
    big = [("u8", rng.integers(0, 60, 300_000).astype(np.uint8)),
           ("bf16", (rng.normal(0, 0.02, 200_000).astype(np.float32).view(np.uint32) >> 16)
            .astype(np.uint16))]
    small = [("u8", rng.integers(0, 9, 70_000).astype(np.uint8))]
    s = torch.cuda.Stream(dev)
    cap, wsb = wc.encode_device_bounds([(e[0], e[1].nbytes) for e in big])
    blob = torch.full((cap,), 0xA5, dtype=torch.uint8, device=dev)
    ws = torch.empty(wsb, dtype=torch.uint8, device=dev)
    size = torch.zeros(1, dtype=torch.int64, device=dev)
    for entries in (big, small):
        dents = [(e[0], to_dev(e[1], dev)) for e in entries]
        torch.cuda.synchronize()
        with torch.cuda.stream(s):
            wc.encode_device(dents, blob=blob, workspace=ws, size=size, stream=s)
        s.synchronize()
        n = int(size.item())
        assert blob[:n].cpu().numpy().tobytes() == oracle.encode(entries)
    first_n = len(oracle.encode(big))
    assert bool((blob[first_n:] == 0xA5).all())


def test_argument_errors(dev):
    x = to_dev(np.arange(4096, dtype=np.uint8), dev)
    cap, wsb = wc.encode_device_bounds([("u8", x)])
    blob = torch.empty(cap, dtype=torch.uint8, device=dev)
    ws = torch.empty(wsb, dtype=torch.uint8, device=dev)
    with pytest.raises(wc.WcError):      # blob capacity one byte short
        wc.encode_device([("u8", x)], blob=blob[: cap - 1], workspace=ws)
    with pytest.raises(wc.WcError):      # workspace too small
        wc.encode_device([("u8", x)], blob=blob, workspace=ws[:16])
    big = torch.empty(8192, dtype=torch.uint8, device=dev)
    with pytest.raises(wc.WcError):      # misaligned source
        wc.encode_device([("u8", big[1:4097])], blob=blob, workspace=ws)
    with pytest.raises(wc.WcError):      # odd byte count of a 16-bit format
        wc.encode_device([("bf16", x[:4095])])
    with pytest.raises(wc.WcError):
        wc.analyze_device("bf16", big[1:4097])


# --- analysis ---------------------------------------------------------------

def _same_stats(got, want):
    assert got["n_fields"] == want["n_fields"]
    assert got["count"] == want["count"]
    for a, b in zip(got["hist"], want["hist"]):
        assert np.array_equal(a, b)
    assert got["H"] == pytest.approx(want["H"], rel=0, abs=1e-12)
    if np.isnan(want["H_joint16"]):
        assert np.isnan(got["H_joint16"])
    else:
        assert got["H_joint16"] == pytest.approx(want["H_joint16"], rel=0, abs=1e-12)
    assert got["bound_bytes"] == pytest.approx(want["bound_bytes"], rel=1e-13)


@pytest.mark.parametrize("cfg,div", [(1, 1), (3, 4), (4, 4), (6, 4), (7, 4)])
def test_analyze_device_matches_oracle(dev, cfg, div):
    for t in synth.config(cfg, div=div)[:4]:
        got = wc.analyze_device(t.dtype, to_dev(t.data, dev))
        _same_stats(got, oracle.analyze(t.dtype, t.data))
        host = wc.analyze(t.dtype, t.data)
        assert got["H"] == host["H"] and got["bound_bytes"] == host["bound_bytes"]


def test_analyze_device_edges(dev):
    rng = np.random.default_rng(3)
    allw = rng.permutation(np.arange(65536, dtype=np.uint32)).astype(np.uint16)
    cases = [("bf16", allw), ("fp16", allw[:3]), ("u8", np.arange(256, dtype=np.uint8)),
             ("u4", rng.integers(0, 256, 17).astype(np.uint8)), ("u8", np.zeros(0, np.uint8)),
             ("bf16", np.zeros(0, np.uint16)), ("u8", np.full(1000, 7, np.uint8))]
    for dt, d in cases:
        x = to_dev(d, dev) if d.size else torch.empty(0, dtype=torch.uint8, device=dev)
        _same_stats(wc.analyze_device(dt, x), oracle.analyze(dt, d))


def _records_match_oracle(raw, t, host, rng, n_sample=3):
    """For tensor t of a blob of bf16 tensors (64 lanes, flat 64 KiB chunks):
    its frequency table is the oracle's normalisation of the oracle's
    histogram of the whole tensor; sampled chunk records (the first, the last,
    and random ones) are byte for byte the oracle's encode of that chunk's
    symbols; and the oracle decodes those chunks back to the original bytes."""
    d = 64 + 96 * t
    first = struct.unpack_from("<Q", raw, d + 24)[0]
    n_chunks = struct.unpack_from("<Q", raw, d + 32)[0]
    freq_off = struct.unpack_from("<Q", raw, d + 48)[0]
    index_off = struct.unpack_from("<Q", raw, 32)[0]
    coded, _ = oracle.symbols("bf16", host)
    freq = oracle.normalise(oracle.histogram(coded))
    assert np.array_equal(np.frombuffer(raw[freq_off:freq_off + 512].tobytes(), np.uint16), freq)
    E = 65536 // 2
    picks = sorted({0, n_chunks - 1} | set(rng.choice(n_chunks, n_sample, replace=False).tolist()))
    out = np.empty(host.size * 2, np.uint8)
    orig = host.view(np.uint8).reshape(-1)
    for c in picks:
        # an untiled bf16 chunk: each lane starts at 2^16 plus its first two
        # exponent bytes (the first lowest), which are not coded
        sym = coded[c * E:(c + 1) * E]
        init = [(1 << 16) + sum(int(sym[lane * 8 + t]) << (8 * t) for t in range(2)
                                if lane * 8 + t < sym.size) for lane in range(64)]
        states, words = oracle.encode_stream(sym, freq, 64, 8, init=np.array(init, np.uint32),
                                             skip=2)
        off = 16 * struct.unpack_from("<I", raw, index_off + 4 * (first + c))[0]
        nw, na, nsym, zero = struct.unpack_from("<IIII", raw, off)
        assert (nw, na, zero) == (words.size, states.size, 0), (t, c)
        assert nsym == min(E, coded.size - c * E), (t, c)
        got_states = np.frombuffer(raw[off + 16:off + 16 + 4 * na].tobytes(), np.uint32)
        w0 = off + 16 + (4 * na + 15) // 16 * 16
        got_words = np.frombuffer(raw[w0:w0 + 2 * nw].tobytes(), np.uint16)
        assert np.array_equal(got_states, states) and np.array_equal(got_words, words), (t, c)
        oracle.decode_chunks(raw, t, c, c + 1, out=out)
        lo, hi = 2 * c * E, min(2 * (c + 1) * E, out.size)
        assert np.array_equal(out[lo:hi], orig[lo:hi]), (t, c)


@pytest.mark.parametrize("model", list(synth.MODEL_LAYERS))
def test_model_family_layer(dev, model):
    """A whole bf16 decoder layer of each model family of the paper (1.5B to
    405B parameters; the benchmark's sweep draw), at its real shapes.  The
    device encoder's blob decodes on the GPU to the layer, bit for bit.
    Against the oracle: for the two smallest families the whole blob equals
    the oracle's encode; for every family each tensor's table equals the
    oracle's, sampled chunk records equal the oracle's encode of those chunks,
    and the oracle decodes them back to the original bytes."""
    say("model layer", model)
    shapes, sigma = synth.MODEL_LAYERS[model]
    seed = 20 + list(synth.MODEL_LAYERS).index(model)
    tens = synth.layer_torch_device(shapes, sigma, seed, device="cuda")
    dents = [("bf16", t, shape) for _, t, shape in tens]
    blob, size = wc.encode_device(dents)
    torch.cuda.synchronize()
    n = int(size.item())
    raw = blob[:n].cpu().numpy()
    desc = wc.open_blob(raw)
    err = torch.zeros(1, dtype=torch.int32, device=dev)
    outs = wc.decode_torch(desc, blob, err=err)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    for (_, t, _), out in zip(tens, outs):
        assert torch.equal(out, t)
    del outs
    say(f"  {model}: {n / 1e9:.3f} GB blob, {sum(t.numel() for _, t, _ in tens) / 1e9:.3f} GB "
        "decoded bit-exact on the GPU")
    rng = np.random.default_rng(seed)
    host = []
    for j, (name, t, shape) in enumerate(tens):
        h = t.cpu().numpy().view(np.uint16)
        _records_match_oracle(raw, j, h, rng)
        if model in ("qwen2-1.5b", "mistral-7b"):
            host.append(("bf16", h, shape))
        say(f"  {model} {name} {shape}: table and sampled records equal the oracle's")
    if host:
        assert raw.tobytes() == oracle.encode(host)
    del tens, blob
    torch.cuda.empty_cache()
