"""wc_decode, wc_gemv, wc_gemm (with its x packing), wc_gemm_i8, wc_gemv_mx,
wc_gemv_w4 and wc_encode_device only launch kernels on the caller's stream: no allocation,
no memset node, no synchronisation.  So a HIP graph can capture them, the way
a serving loop replays one step.

Each test captures the calls once and replays the graph several times.
Between replays the outputs are overwritten eagerly and the device is
synchronised.  Every replay is checked against the oracle: decoded bytes equal
the original tensors, small-integer products equal the oracle's exact product,
and device blobs equal the oracle's encoder byte for byte.  The outputs and the
error word are cleared inside the graph by fill kernels (torch's zero_()).
"""
import numpy as np
import pytest

import oracle
from paper_2606_15789_amd import synth, wc

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

REPLAYS = 3


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda:0")


def say(*a):
    print(*a, flush=True)


def _bf16(a):
    return (np.asarray(a, np.float32).view(np.uint32) >> 16).astype(np.uint16)


def _dev_bf16(bits, dev):
    return torch.from_numpy(bits.view(np.int16)).to(dev).view(torch.bfloat16)


def _capture(dev, body):
    """Warm up `body` on a side stream, then capture it into a graph."""
    side = torch.cuda.Stream(dev)
    side.wait_stream(torch.cuda.current_stream(dev))
    with torch.cuda.stream(side):
        body()
    torch.cuda.current_stream(dev).wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        body()
    torch.cuda.synchronize()
    return g


def test_decode_replayed_from_a_graph(dev):
    """One decode launch over the int8 layer (int8 codes, fp16 scales, bf16
    norms) and a tiled bf16 matrix, captured and replayed."""
    say("graph: decode")
    ts = synth.config(4, div=8)
    rng = np.random.default_rng(71)
    w = _bf16(rng.normal(0, 0.02, (256, 2048)))
    entries = [(t.dtype, t.data) for t in ts] + [("bf16", w, w.shape)]
    blob = wc.encode(entries, tile=(64, 512), tile_order=1)
    want = [torch.from_numpy(np.ascontiguousarray(e[1]).view(np.uint8).reshape(-1).copy()).to(dev)
            for e in entries]
    raw = blob.tobytes()
    ref = oracle.decode(raw)
    for r, e in zip(ref, entries):
        assert np.array_equal(r, np.ascontiguousarray(e[1]).view(np.uint8).reshape(-1))
    d = wc.to_device(blob, dev)
    outs = [torch.empty(n, dtype=torch.uint8, device=dev) for n in blob.out_bytes]
    err = torch.zeros(1, dtype=torch.int32, device=dev)

    def body():
        err.zero_()
        wc.decode_torch(blob, d, outs, err=err)

    g = _capture(dev, body)
    for k in range(REPLAYS):
        for o in outs:
            o.fill_(0x5A + k)
        err.fill_(0)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert int(err.item()) == 0, (k, wc.describe_errors(int(err.item())))
        for t, (o, x) in enumerate(zip(outs, want)):
            assert torch.equal(o, x), (k, t)


def test_fused_gemms_replayed_from_a_graph(dev):
    """wc_gemv (16-row MFMA tiles, 8 rows of x), wc_gemm (64-row tiles, 100
    rows: x packing + shared GEMM), wc_gemm_i8 (16 rows), wc_gemv_mx (MXFP4,
    8 rows) and wc_gemv_w4 (int4 with zero points, 8 rows), all in one graph, on small integers so that every replay must
    equal the exact product."""
    say("graph: fused GEMMs")
    rng = np.random.default_rng(72)
    w = _bf16(rng.integers(-4, 5, (128, 1024)).astype(np.float32))
    wi = rng.integers(-128, 128, (64, 1024)).astype(np.int8)
    b16 = wc.encode([("bf16", w, w.shape)], tile=(16, 1024), tile_order=1)
    b64 = wc.encode([("bf16", w, w.shape)], tile=(64, 512), tile_order=1)
    bi8 = wc.encode([("u8", wi, wi.shape)], tile=(16, 256), tile_order=1)
    x8 = _bf16(rng.integers(-3, 4, (8, 1024)).astype(np.float32))
    x100 = _bf16(rng.integers(-3, 4, (100, 1024)).astype(np.float32))
    xi = rng.integers(-128, 128, (16, 1024)).astype(np.int8)
    ref8, _ = oracle.gemv_bf16(w, x8)
    ref100, _ = oracle.gemv_bf16(w, x100)
    refi = oracle.gemm_i8(wi, xi)
    # int4 with zero points at scale 1 (binary16 0x3C00)
    c4 = rng.integers(0, 16, (32, 1024)).astype(np.uint8)
    z4 = rng.integers(0, 16, (32, 8)).astype(np.uint8)
    p4 = (c4[:, 0::2] | (c4[:, 1::2] << 4)).astype(np.uint8)
    bw4 = wc.encode([("u8", p4, (32, 512))], tile=(16, 256), tile_order=1)
    s4 = torch.full((32 * 8,), 0x3C00, dtype=torch.int16, device=dev)
    dz4 = torch.from_numpy(z4.reshape(-1).copy()).to(dev)
    ref4, _ = oracle.gemv_int4(p4, np.full((32, 8), 0x3C00, np.uint16), z4, x8)
    # MXFP4: e2m1 integers at scale 1 (e8m0 127)
    table = {0: 0, 1: 2, 2: 4, 3: 5, 4: 6, 6: 7}
    vals = rng.choice([0, 1, 2, 3, 4, 6, -1, -2, -3, -4, -6], (32, 1024))
    codes = np.vectorize(lambda v: table[abs(v)] | (8 if v < 0 else 0))(vals).astype(np.uint8)
    bmx = wc.encode([("fp4_e2m1", codes[:, 0::2] | (codes[:, 1::2] << 4), codes.shape)],
                    tile=(16, 512), tile_order=1)
    smx = torch.full((32 * 1024 // 32,), 127, dtype=torch.uint8, device=dev)
    refmx, _ = oracle.gemv_mxfp4(codes[:, 0::2] | (codes[:, 1::2] << 4),
                                 np.full((32, 32), 127, np.uint8), x8)
    assert np.array_equal(refmx, (x8.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
                          @ vals.T.astype(np.float64))
    d16, d64, di8 = wc.to_device(b16, dev), wc.to_device(b64, dev), wc.to_device(bi8, dev)
    dmx = wc.to_device(bmx, dev)
    dw4 = wc.to_device(bw4, dev)
    dx8, dx100 = _dev_bf16(x8, dev), _dev_bf16(x100, dev)
    dxi = torch.from_numpy(xi).to(dev)
    y8 = torch.empty((8, 128), dtype=torch.float32, device=dev)
    y100 = torch.empty((100, 128), dtype=torch.float32, device=dev)
    yi = torch.empty((16, 64), dtype=torch.int32, device=dev)
    ymx = torch.empty((8, 32), dtype=torch.float32, device=dev)
    y4 = torch.empty((8, 32), dtype=torch.float32, device=dev)
    need = wc.gemm_workspace_bytes(b64, [0], [dx100.data_ptr()], 100)
    ws = torch.empty(max(need, 256), dtype=torch.uint8, device=dev)
    err = torch.zeros(1, dtype=torch.int32, device=dev)

    def body():
        err.zero_()
        y8.zero_()
        y100.zero_()
        yi.zero_()
        ymx.zero_()
        y4.zero_()
        wc.gemv_torch(b16, d16, [0], [dx8], ys=[y8], err=err)
        wc.gemv_w4_torch(bw4, dw4, [0], [s4], [dz4], [dx8], ys=[y4], err=err)
        wc.gemv_mx_torch(bmx, dmx, [0], [smx], [dx8], ys=[ymx], err=err)
        wc.gemm_torch(b64, d64, [0], [dx100], ys=[y100], workspace=ws, err=err)
        wc.gemm_i8_torch(bi8, di8, [0], [dxi], ys=[yi], err=err)

    g = _capture(dev, body)
    for k in range(REPLAYS):
        y8.fill_(float("nan"))
        y100.fill_(float("nan"))
        yi.fill_(-7)
        ymx.fill_(float("nan"))
        y4.fill_(float("nan"))
        ws.fill_(0xEE)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert int(err.item()) == 0, (k, wc.describe_errors(int(err.item())))
        assert np.array_equal(y8.cpu().numpy().astype(np.float64), ref8), k
        assert np.array_equal(y100.cpu().numpy().astype(np.float64), ref100), k
        assert np.array_equal(yi.cpu().numpy().astype(np.int64), refi), k
        assert np.array_equal(ymx.cpu().numpy().astype(np.float64), refmx), k
        assert np.array_equal(y4.cpu().numpy().astype(np.float64), ref4), k


def test_device_encoder_replayed_from_a_graph(dev):
    """wc_encode_device (histogram clears, counts, table normalisation, chunk
    encode, index scan, packing) captured once; each replay re-encodes tensors
    whose contents changed in place since the capture, and must write the
    oracle's blob for the new contents."""
    say("graph: device encoder")
    rng = np.random.default_rng(73)
    shapes = [("bf16", 300_000), ("u8", 150_001), ("u4", 70_000)]

    def draw(k):
        out = []
        for dt, n in shapes:
            if dt == "bf16":
                out.append((dt, _bf16(rng.normal(0, 0.02 * (k + 1), n))))
            else:
                out.append((dt, rng.integers(0, 60 + 40 * k, n).astype(np.uint8)))
        return out

    first = draw(0)
    dents = [(dt, torch.from_numpy(np.ascontiguousarray(a).view(np.uint8).reshape(-1).copy()).to(dev))
             for dt, a in first]
    cap, wsb = wc.encode_device_bounds(dents)
    blob = torch.empty(cap, dtype=torch.uint8, device=dev)
    ws = torch.empty(wsb, dtype=torch.uint8, device=dev)
    size = torch.zeros(1, dtype=torch.int64, device=dev)

    def body():
        wc.encode_device(dents, blob=blob, workspace=ws, size=size)

    g = _capture(dev, body)
    for k in range(REPLAYS):
        host = draw(k + 1)
        for (dt, x), (_, a) in zip(dents, host):
            x.copy_(torch.from_numpy(np.ascontiguousarray(a).view(np.uint8).reshape(-1).copy()))
        blob.fill_(0xA5)
        ws.fill_(0x3C)
        size.fill_(0)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        n = int(size.item())
        assert blob[:n].cpu().numpy().tobytes() == oracle.encode(host), k
