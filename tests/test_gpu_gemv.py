"""GPU parity of the fused decode-GEMM (wc_gemv) and of column-block tiles.

wc_gemv adds x * W^T to y, decoding W on the fly.  The reference is the
oracle's fp64 product of the same bf16 values (orc_gemv_bf16, pinned on
one-hot and small-integer inputs).  The GPU sums in fp32 (v_dot2_f32_bf16 or
v_mfma_f32_32x32x16_bf16 for 64-row tiles, v_mfma_f32_32x32x16_bf16 for 32-row
and v_mfma_f32_16x16x32_bf16 for 16-row tiles, then fp32 atomics across the
tiles or tile segments of a row band); bf16 products are exact in fp32, so with at
most K roundings of relative size 2^-24 each, |y - y_ref| <= K * 2^-24 *
sum_k |x_k w_k|.  The test allows twice that.
"""
import struct

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


def _bf16(a):
    return (np.asarray(a, np.float32).view(np.uint32) >> 16).astype(np.uint16)


def _dev_x(x_bits, dev):
    return torch.from_numpy(x_bits.view(np.int16)).to(dev).view(torch.bfloat16)


def _run_gemv(blob, dev, t, x_bits, y0=None, expect_err=0):
    d = wc.to_device(blob, dev)
    err = torch.zeros(1, dtype=torch.int32, device=dev)
    ys = None if y0 is None else [torch.from_numpy(y0).to(dev)]
    ys = wc.gemv_torch(blob, d, [t], [_dev_x(x_bits, dev)], ys=ys, err=err)
    torch.cuda.synchronize()
    assert int(err.item()) == expect_err, wc.describe_errors(int(err.item()))
    return ys[0].cpu().numpy().astype(np.float64)


def _run_gemm(blob, dev, t, x_bits, expect_err=0):
    d = wc.to_device(blob, dev)
    err = torch.zeros(1, dtype=torch.int32, device=dev)
    ys = wc.gemm_torch(blob, d, [t], [_dev_x(x_bits, dev)], err=err)
    torch.cuda.synchronize()
    assert int(err.item()) == expect_err, wc.describe_errors(int(err.item()))
    return ys[0].cpu().numpy().astype(np.float64)


def _check(y, w, x, scale=1.0):
    ref, absref = oracle.gemv_bf16(w, x)
    K = w.shape[1]
    tol = 2.0 * K * 2.0 ** -24 * absref * scale + 1e-30
    bad = np.abs(y - scale * ref) > tol
    assert not bad.any(), (np.argwhere(bad)[:5], float(np.abs(y - scale * ref).max()))


@pytest.mark.parametrize("tile", [(64, 256), (64, 512), (32, 128)])
@pytest.mark.parametrize("lanes", [64, 32])
def test_column_block_tiles_decode_exactly(dev, tile, lanes):
    say("column blocks", tile, "lanes", lanes)
    ts = synth.config(2, div=8)
    pairs = [(t.dtype, t.data, t.shape if len(t.shape) == 2 else None) for t in ts]
    blob = wc.encode(pairs, lanes=lanes, tile=tile, tile_order=1)
    assert any(i["tile_order"] == 1 for i in oracle.tensor_info(blob.tobytes()))
    d = wc.to_device(blob, dev)
    err = torch.zeros(1, dtype=torch.int32, device=dev)
    outs = wc.decode_torch(blob, d, err=err)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    ref = oracle.decode(blob.tobytes())
    for (_, data, _), o, r in zip(pairs, outs, ref):
        got = o.cpu().numpy()
        assert np.array_equal(got, np.ascontiguousarray(data).view(np.uint8).reshape(-1))
        assert np.array_equal(got, r)


@pytest.mark.parametrize("shape,tile", [((256, 512), (64, 256)), ((192, 1024), (64, 512)),
                                        ((1024, 4096), (64, 512)), ((64, 256), (64, 256))])
@pytest.mark.parametrize("m", [1, 3, 5, 6, 8])
def test_gemv_matches_the_reference(dev, shape, tile, m):
    say("gemv", shape, tile, m)
    rng = np.random.default_rng(shape[0] + m)
    w = _bf16(rng.normal(0, 0.02, shape))
    x = _bf16(rng.normal(0, 1.0, (m, shape[1])))
    blob = wc.encode([("bf16", w, shape)], tile=tile, tile_order=1)
    y = _run_gemv(blob, dev, 0, x)
    _check(y, w, x)


def test_gemv_adds_to_y_and_picks_the_tensor(dev):
    rng = np.random.default_rng(21)
    w0 = _bf16(rng.normal(0, 0.02, (128, 512)))
    w1 = _bf16(rng.normal(0, 0.05, (256, 1024)))
    norm = _bf16(rng.normal(1, 0.02, 512))
    blob = wc.encode([("bf16", norm), ("bf16", w0, (128, 512)), ("bf16", w1, (256, 1024))],
                     tile=(64, 512), tile_order=1, codebook="layer")
    x = _bf16(rng.normal(0, 1.0, (2, 1024)))
    y = _run_gemv(blob, dev, 2, x)
    _check(y, w1, x)
    ref, _ = oracle.gemv_bf16(w1, x)
    y2 = _run_gemv(blob, dev, 2, x, y0=ref.astype(np.float32))    # y += x W^T
    _check(y2, w1, x, scale=2.0)
    x0 = np.ascontiguousarray(x[:, :512])
    _check(_run_gemv(blob, dev, 1, x0), w0, x0)


def test_gemv_full_size_projection(dev):
    """A Llama-3-70B q_proj (8192 x 8192) in 64 x 512 column-block tiles."""
    w = synth.config(5)[0].data
    assert w.shape == (8192, 8192)
    blob = wc.encode([("bf16", w, (8192, 8192))], tile=(64, 512), tile_order=1)
    x = _bf16(np.random.default_rng(22).normal(0, 1.0, (4, 8192)))
    y = _run_gemv(blob, dev, 0, x)
    _check(y, w, x)


@pytest.mark.parametrize("tiles,m", [(6144, 16), (6145, 1), (8192, 16), (8193, 16), (7000, 17)])
def test_gemv_bf16_around_the_wide_kernels_window(dev, tiles, m):
    """bf16 weights on 16-row tiles run on a 16-wave kernel when the launch has
    one block of x rows (m <= 16) and its tiles overflow the 8-wave kernel's
    resident waves (6144 on a 256-CU MI355X) but fit the 16-wave kernel's
    (8192).  Tile counts on both edges of that window and m = 17 (outside it):
    sampled rows of y within the fp32 summation bound of the oracle's
    product."""
    say("bf16 wide window", tiles, m)
    rows, cols = 16 * tiles, 512
    rng = np.random.default_rng(tiles + 1)
    w = _bf16(rng.standard_normal((rows, cols), dtype=np.float32) * np.float32(0.02))
    blob = wc.encode([("bf16", w, w.shape)], tile=(16, 512), tile_order=1)
    x = _bf16(rng.normal(0, 1.0, (m, cols)))
    y = _run_gemv(blob, dev, 0, x)
    pick = np.concatenate([rng.choice(rows, 64, replace=False), [0, rows - 1]])
    _check(y[:, pick], np.ascontiguousarray(w[pick]), x)


def test_gemv_reports_corruption(dev):
    rng = np.random.default_rng(23)
    w = _bf16(rng.normal(0, 0.02, (128, 512)))
    blob = wc.encode([("bf16", w, (128, 512))], tile=(64, 256), tile_order=1)
    raw = blob.tobytes()
    idx = struct.unpack_from("<Q", raw, 32)[0]
    off1 = struct.unpack_from("<I", raw, idx + 4)[0] * 16
    d = wc.to_device(blob, dev)
    d[off1 + 16 + 20] ^= 0x01                      # a lane state of tile 1
    x = _dev_x(_bf16(rng.normal(0, 1, (1, 512))), dev)
    err = torch.zeros(1, dtype=torch.int32, device=dev)
    wc.gemv_torch(blob, d, [0], [x], err=err)
    torch.cuda.synchronize()
    assert int(err.item()) & 0x6


def test_fused_gemms_on_a_side_stream(dev):
    """wc_gemv, wc_gemm (shared path) and wc_gemm_i8 issued on a non-default
    stream, with the inputs made on that stream: every launch, the x packing
    included, follows the stream's order."""
    rng = np.random.default_rng(61)
    w = _bf16(rng.normal(0, 0.02, (128, 1024)))
    wi = rng.integers(-128, 128, (64, 1024)).astype(np.int8)
    b16 = wc.encode([("bf16", w, w.shape)], tile=(16, 1024), tile_order=1)
    b64 = wc.encode([("bf16", w, w.shape)], tile=(64, 512), tile_order=1)
    bi8 = wc.encode([("u8", wi, wi.shape)], tile=(16, 256), tile_order=1)
    x16 = _bf16(rng.normal(0, 1.0, (16, 1024)))
    x100 = _bf16(rng.normal(0, 1.0, (100, 1024)))
    xi = rng.integers(-128, 128, (16, 1024)).astype(np.int8)
    side = torch.cuda.Stream(dev)
    with torch.cuda.stream(side):
        d16, d64, di8 = wc.to_device(b16, dev), wc.to_device(b64, dev), wc.to_device(bi8, dev)
        y16 = wc.gemv_torch(b16, d16, [0], [_dev_x(x16, dev)], stream=side)[0]
        y100 = wc.gemm_torch(b64, d64, [0], [_dev_x(x100, dev)], stream=side)[0]
        yi = wc.gemm_i8_torch(bi8, di8, [0], [torch.from_numpy(xi).to(dev)], stream=side)[0]
    side.synchronize()
    _check(y16.cpu().numpy().astype(np.float64), w, x16)
    _check(y100.cpu().numpy().astype(np.float64), w, x100)
    assert np.array_equal(yi.cpu().numpy().astype(np.int64), oracle.gemm_i8(wi, xi))


@pytest.mark.parametrize("m", [1, 5, 100])
def test_gemv_many_jobs_in_one_launch(dev, m):
    """Every projection of a scaled 8B layer in one call; jobs with the same K
    share one x, as q/k/v and gate/up do in a transformer layer."""
    ts = [t for t in synth.config(2, div=4) if len(t.shape) == 2]
    blob = wc.encode([(t.dtype, t.data, t.shape) for t in ts], tile=(64, 256), tile_order=1,
                     codebook="layer")
    d = wc.to_device(blob, dev)
    rng = np.random.default_rng(31 + m)
    xbits = {}
    for t in ts:
        xbits.setdefault(t.shape[1], _bf16(rng.normal(0, 1.0, (m, t.shape[1]))))
    xdev = {k: _dev_x(v, dev) for k, v in xbits.items()}
    err = torch.zeros(1, dtype=torch.int32, device=dev)
    ys = wc.gemm_torch(blob, d, list(range(len(ts))), [xdev[t.shape[1]] for t in ts], err=err)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    for t, y in zip(ts, ys):
        _check(y.cpu().numpy().astype(np.float64), t.data, xbits[t.shape[1]])


# --- 16-row column-block tiles: the product on the matrix cores --------------

@pytest.mark.parametrize("shape,tile", [((256, 512), (16, 256)), ((192, 1024), (16, 512)),
                                        ((1024, 4096), (16, 2048)), ((16, 256), (16, 256)),
                                        ((256, 512), (32, 256)), ((192, 1024), (32, 1024)),
                                        ((32, 128), (32, 128)), ((256, 512), (64, 256)),
                                        ((192, 1024), (64, 512)), ((64, 128), (64, 16))])
@pytest.mark.parametrize("m", [1, 3, 16, 17, 33, 64])
def test_mfma_gemm_matches_the_reference(dev, shape, tile, m):
    say("mfma gemm", shape, tile, m)
    rng = np.random.default_rng(shape[0] + 7 * m)
    w = _bf16(rng.normal(0, 0.02, shape))
    x = _bf16(rng.normal(0, 1.0, (m, shape[1])))
    blob = wc.encode([("bf16", w, shape)], tile=tile, tile_order=1)
    y = _run_gemv(blob, dev, 0, x)
    _check(y, w, x)


@pytest.mark.parametrize("rows", [16, 32, 64])
@pytest.mark.parametrize("m", [5, 6, 37])
def test_mfma_gemm_small_integers_exact(dev, rows, m):
    """Small-integer x and W (exact in bf16, sums exact in fp32): y must equal
    the oracle's product exactly, which pins the operand and output layouts
    (64-row tiles: the VALU dot products at m = 5, the matrix cores above)."""
    rng = np.random.default_rng(41)
    shape = (64, 512)
    w = _bf16(rng.integers(-4, 5, shape).astype(np.float32))
    x = _bf16(rng.integers(-3, 4, (m, shape[1])).astype(np.float32))
    blob = wc.encode([("bf16", w, shape)], tile=(rows, 256), tile_order=1)
    y = _run_gemv(blob, dev, 0, x)
    ref, _ = oracle.gemv_bf16(w, x)
    assert np.array_equal(y, ref)


@pytest.mark.parametrize("tile", [(16, 2048), (32, 1024), (64, 512)])
def test_mfma_gemm_full_size_layer(dev, tile):
    """All seven projections of a Llama-3-70B layer (numpy draw) in 64 KiB
    tiles, one launch, 64 rows of x: every y within the fp32 bound."""
    ts = synth.config(5)
    blob = wc.encode([(t.dtype, t.data, t.shape) for t in ts], tile=tile, tile_order=1)
    d = wc.to_device(blob, dev)
    rng = np.random.default_rng(42)
    xbits = {}
    for t in ts:
        xbits.setdefault(t.shape[1], _bf16(rng.normal(0, 1.0, (64, t.shape[1]))))
    xdev = {k: _dev_x(v, dev) for k, v in xbits.items()}
    err = torch.zeros(1, dtype=torch.int32, device=dev)
    ys = wc.gemv_torch(blob, d, list(range(len(ts))), [xdev[t.shape[1]] for t in ts], err=err)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    for t, y in zip(ts, ys):
        # rows of W sampled (the fp64 reference of all 8192 x 8192 is slow)
        rows = np.random.default_rng(t.shape[0]).choice(t.shape[0], 64, replace=False)
        ref, absref = oracle.gemv_bf16(np.ascontiguousarray(t.data[rows]), xbits[t.shape[1]])
        tol = 2.0 * t.shape[1] * 2.0 ** -24 * absref + 1e-30
        got = y.cpu().numpy().astype(np.float64)[:, rows]
        assert (np.abs(got - ref) <= tol).all(), t.name


def test_gemv_row_limits(dev):
    """Up to 64 rows of x on 16-row tiles (65 are refused); 64-row tiles take the
    VALU dot products up to 5 rows and the matrix cores above, and 64-row tiles
    narrower than 16 columns take at most 5."""
    rng = np.random.default_rng(43)
    w = _bf16(rng.normal(0, 0.02, (128, 512)))
    b64 = wc.encode([("bf16", w, (128, 512))], tile=(64, 256), tile_order=1)
    b16 = wc.encode([("bf16", w, (128, 512))], tile=(16, 256), tile_order=1)
    narrow = wc.encode([("bf16", w, (128, 512))], tile=(64, 8), tile_order=1)
    x5, x6, x64 = (_bf16(rng.normal(0, 1.0, (m, 512))) for m in (5, 6, 64))
    _check(_run_gemv(b64, dev, 0, x5), w, x5)
    _check(_run_gemv(b64, dev, 0, x6), w, x6)
    _check(_run_gemv(b64, dev, 0, x64), w, x64)
    _check(_run_gemv(b16, dev, 0, x6), w, x6)
    _check(_run_gemv(narrow, dev, 0, x5), w, x5)
    with pytest.raises(wc.WcError):
        _run_gemv(narrow, dev, 0, x6)
    with pytest.raises(wc.WcError):                 # 16-row tiles: at most 64 rows
        _run_gemv(b16, dev, 0, _bf16(rng.normal(0, 1.0, (65, 512))))


# --- many rows of x: wc_gemm, the shared fused GEMM on 64-row tiles ----------
# The waves of a workgroup decode up to 8 tiles of one band once and multiply
# every decoded pair of wave rows by their own 32 rows of packed x (256 per pass).

@pytest.mark.parametrize("shape,tile", [((128, 5120), (64, 512)),   # 10 tiles: 2 + 6 idle waves
                                        ((64, 4096), (64, 512)),    # one full segment
                                        ((192, 1024), (64, 256)),   # 4 tiles, 4 idle waves
                                        ((64, 128), (64, 16)),      # one pair per tile
                                        ((128, 9216), (64, 512))])  # 18 tiles: 3 segments
@pytest.mark.parametrize("m", [65, 100, 256, 300])
def test_shared_gemm_matches_the_reference(dev, shape, tile, m):
    say("shared gemm", shape, tile, m)
    rng = np.random.default_rng(shape[1] + m)
    w = _bf16(rng.normal(0, 0.02, shape))
    x = _bf16(rng.normal(0, 1.0, (m, shape[1])))
    blob = wc.encode([("bf16", w, shape)], tile=tile, tile_order=1)
    _check(_run_gemm(blob, dev, 0, x), w, x)


@pytest.mark.parametrize("m", [65, 513, 1000])
def test_shared_gemm_small_integers_exact(dev, m):
    """Exact small-integer products pin the operand exchange through LDS, the
    x blocks of every wave and the passes over x."""
    rng = np.random.default_rng(44 + m)
    shape = (128, 5120)
    w = _bf16(rng.integers(-4, 5, shape).astype(np.float32))
    x = _bf16(rng.integers(-3, 4, (m, shape[1])).astype(np.float32))
    blob = wc.encode([("bf16", w, shape)], tile=(64, 512), tile_order=1)
    y = _run_gemm(blob, dev, 0, x)
    ref, _ = oracle.gemv_bf16(w, x)
    assert np.array_equal(y, ref)


def test_shared_gemm_full_size_layer(dev):
    """All seven projections of a Llama-3-70B layer (numpy draw), 64 x 512
    tiles, 256 rows of x, one launch: sampled y within the fp32 bound."""
    ts = synth.config(5)
    blob = wc.encode([(t.dtype, t.data, t.shape) for t in ts], tile=(64, 512), tile_order=1)
    d = wc.to_device(blob, dev)
    rng = np.random.default_rng(45)
    xbits = {}
    for t in ts:
        xbits.setdefault(t.shape[1], _bf16(rng.normal(0, 1.0, (256, t.shape[1]))))
    xdev = {k: _dev_x(v, dev) for k, v in xbits.items()}
    err = torch.zeros(1, dtype=torch.int32, device=dev)
    ys = wc.gemm_torch(blob, d, list(range(len(ts))), [xdev[t.shape[1]] for t in ts], err=err)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    for t, y in zip(ts, ys):
        rows = np.random.default_rng(t.shape[0]).choice(t.shape[0], 32, replace=False)
        xr = xbits[t.shape[1]][::8]                      # 32 of the 256 x rows
        ref, absref = oracle.gemv_bf16(np.ascontiguousarray(t.data[rows]), xr)
        tol = 2.0 * t.shape[1] * 2.0 ** -24 * absref + 1e-30
        got = y.cpu().numpy().astype(np.float64)[::8][:, rows]
        assert (np.abs(got - ref) <= tol).all(), t.name


def test_shared_gemm_reports_corruption(dev):
    """A bad lane state and a bad index entry: the launch completes (the wave
    with the bad entry still takes part in every exchange) and reports both."""
    rng = np.random.default_rng(46)
    w = _bf16(rng.normal(0, 0.02, (128, 5120)))
    blob = wc.encode([("bf16", w, (128, 5120))], tile=(64, 512), tile_order=1)
    raw = blob.tobytes()
    idx = struct.unpack_from("<Q", raw, 32)[0]
    x = _dev_x(_bf16(rng.normal(0, 1, (100, 5120))), dev)
    off1 = struct.unpack_from("<I", raw, idx + 4)[0] * 16
    d = wc.to_device(blob, dev)
    d[off1 + 16 + 20] ^= 0x01                      # a lane state of tile 1
    err = torch.zeros(1, dtype=torch.int32, device=dev)
    wc.gemm_torch(blob, d, [0], [x], err=err)
    torch.cuda.synchronize()
    assert int(err.item()) & 0x6
    d = wc.to_device(blob, dev)
    d[idx + 4 * 3 + 3] = 0x7F                      # index entry of tile 3: far past the records
    err.zero_()
    wc.gemm_torch(blob, d, [0], [x], err=err)
    torch.cuda.synchronize()
    assert int(err.item()) & 0x1


def test_shared_gemm_limits(dev):
    """Past 64 rows of x: 64-row tiles only, all full; at most 4096 rows;
    wc_gemv stops at 64."""
    rng = np.random.default_rng(47)
    w = _bf16(rng.normal(0, 0.02, (128, 512)))
    b16 = wc.encode([("bf16", w, (128, 512))], tile=(16, 256), tile_order=1)
    ragged = wc.encode([("bf16", w[:100], (100, 512))], tile=(64, 256), tile_order=1)
    b64 = wc.encode([("bf16", w, (128, 512))], tile=(64, 256), tile_order=1)
    x65 = _bf16(rng.normal(0, 1.0, (65, 512)))
    for b in (b16, ragged):
        with pytest.raises(wc.WcError) as e:
            _run_gemm(b, dev, 0, x65)
        assert e.value.rc == -5
    with pytest.raises(wc.WcError) as e:
        _run_gemv(b64, dev, 0, x65)
    assert e.value.rc == -1
    _check(_run_gemm(b64, dev, 0, x65), w, x65)
    x4096 = _bf16(rng.normal(0, 1.0, (4096, 512)))
    _check(_run_gemm(b64, dev, 0, x4096), w, x4096)
    with pytest.raises(wc.WcError) as e:
        _run_gemm(b64, dev, 0, _bf16(rng.normal(0, 1.0, (4097, 512))))
    assert e.value.rc == -1


@pytest.mark.parametrize("m", [1, 37, 64])
def test_gemm_up_to_64_rows_is_gemv(dev, m):
    """wc_gemm below 65 rows runs wc_gemv's kernels, with no workspace."""
    rng = np.random.default_rng(48 + m)
    w = _bf16(rng.normal(0, 0.02, (128, 1024)))
    x = _bf16(rng.normal(0, 1.0, (m, 1024)))
    for tile in ((64, 512), (16, 1024)):
        blob = wc.encode([("bf16", w, (128, 1024))], tile=tile, tile_order=1)
        assert wc.gemm_workspace_bytes(blob, [0], [16], m) == 0
        _check(_run_gemm(blob, dev, 0, x), w, x)


def test_gemm_jobs_sharing_x(dev):
    """q, k and v of one x and a second x: one packed copy per distinct x,
    every product right, the workspace used as sized."""
    rng = np.random.default_rng(49)
    ws_ = [_bf16(rng.normal(0, 0.02, (n, 1024))) for n in (256, 64, 64)]
    w2 = _bf16(rng.normal(0, 0.02, (128, 2048)))
    blob = wc.encode([("bf16", w, w.shape) for w in ws_] + [("bf16", w2, w2.shape)],
                     tile=(64, 256), tile_order=1, codebook="layer")
    d = wc.to_device(blob, dev)
    x1 = _bf16(rng.normal(0, 1.0, (130, 1024)))
    x2 = _bf16(rng.normal(0, 1.0, (130, 2048)))
    dx1, dx2 = _dev_x(x1, dev), _dev_x(x2, dev)
    xs = [dx1, dx1, dx1, dx2]
    need = wc.gemm_workspace_bytes(blob, [0, 1, 2, 3], [x.data_ptr() for x in xs], 130)
    assert need == 160 * 1024 * 2 + 160 * 2048 * 2
    ws = torch.empty(need, dtype=torch.uint8, device=dev)
    err = torch.zeros(1, dtype=torch.int32, device=dev)
    ys = wc.gemm_torch(blob, d, [0, 1, 2, 3], xs, workspace=ws, err=err)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    for w, x, y in zip(ws_ + [w2], [x1, x1, x1, x2], ys):
        _check(y.cpu().numpy().astype(np.float64), w, x)


# --- int8 weights, int8 x (W8A8): v_mfma_i32_16x16x64_i8, exact int32 --------

def _run_gemm_i8(blob, dev, t, x, expect_err=0):
    d = wc.to_device(blob, dev)
    err = torch.zeros(1, dtype=torch.int32, device=dev)
    ys = wc.gemm_i8_torch(blob, d, [t], [torch.from_numpy(x).to(dev)], err=err)
    torch.cuda.synchronize()
    assert int(err.item()) == expect_err, wc.describe_errors(int(err.item()))
    return ys[0].cpu().numpy().astype(np.int64)


@pytest.mark.parametrize("shape,tile", [((64, 256), (16, 64)), ((48, 1024), (16, 256)),
                                        ((256, 4096), (16, 4096)), ((32, 64), (16, 16)),
                                        ((16, 2048), (16, 1024))])
@pytest.mark.parametrize("m", [1, 5, 16, 17, 33, 64])
def test_int8_gemm_is_exact(dev, shape, tile, m):
    """Every int32 sum equals the oracle's exact product (tile (16, 16) leaves
    three quarters of each wave row empty: those lanes contribute zero)."""
    say("int8 gemm", shape, tile, m)
    rng = np.random.default_rng(shape[1] + 7 * m)
    w = rng.integers(-128, 128, shape).astype(np.int8)
    x = rng.integers(-128, 128, (m, shape[1])).astype(np.int8)
    blob = wc.encode([("u8", w, shape)], tile=tile, tile_order=1)
    assert np.array_equal(_run_gemm_i8(blob, dev, 0, x), oracle.gemm_i8(w, x))


@pytest.mark.parametrize("tiles,m", [(6144, 16), (6145, 16), (7000, 1), (8192, 16), (8193, 16),
                                     (7000, 17)])
def test_int8_gemm_around_the_wide_kernels_window(dev, tiles, m):
    """wc_gemm_i8 runs on its 16-wave kernel when the launch has one block of x
    rows (m <= 16) and its tiles overflow the 8-wave kernel's resident waves
    (6144 on a 256-CU MI355X) but fit the 16-wave kernel's (8192).  Tile counts
    on both edges of that window, and m = 17 (outside it), give y equal to the
    oracle's int8 product on sampled rows."""
    say("int8 wide window", tiles, m)
    rows, cols = 16 * tiles, 512
    codes = synth.int8_rows_torch_device(rows, cols, 60 + tiles % 89)
    blob = wc.encode([("u8", codes.cpu().numpy(), (rows, cols))], tile=(16, 512), tile_order=1)
    d = wc.to_device(blob, dev)
    x = np.random.default_rng(tiles).integers(-127, 128, (m, cols)).astype(np.int8)
    err = torch.zeros(1, dtype=torch.int32, device=dev)
    y, = wc.gemm_i8_torch(blob, d, [0], [torch.from_numpy(x).to(dev)], err=err)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    w = codes.cpu().numpy().view(np.int8).reshape(rows, cols)
    pick = np.random.default_rng(rows).choice(rows, 64, replace=False)
    pick = np.concatenate([pick, [0, rows - 1]])
    want = oracle.gemm_i8(np.ascontiguousarray(w[pick]), x)
    assert np.array_equal(y.cpu().numpy().astype(np.int64)[:, pick], want)
    del codes, d


def test_int8_gemm_quantised_layer(dev):
    """The int8 projections of the scaled 8B W8 workload (Student-t weights,
    per-row absmax scales) in 16 x 512 tiles, one launch, 16 rows of x."""
    ts = [t for t in synth.config(4, div=4) if t.dtype == "u8" and len(t.shape) == 2]
    assert ts
    blob = wc.encode([(t.dtype, t.data, t.shape) for t in ts], tile=(16, 512), tile_order=1,
                     codebook="layer")
    d = wc.to_device(blob, dev)
    rng = np.random.default_rng(50)
    xs = {}
    for t in ts:
        xs.setdefault(t.shape[1], rng.integers(-127, 128, (16, t.shape[1])).astype(np.int8))
    err = torch.zeros(1, dtype=torch.int32, device=dev)
    ys = wc.gemm_i8_torch(blob, d, list(range(len(ts))),
                          [torch.from_numpy(xs[t.shape[1]]).to(dev) for t in ts], err=err)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    for t, y in zip(ts, ys):
        rows = np.random.default_rng(t.shape[0]).choice(t.shape[0], 48, replace=False)
        want = oracle.gemm_i8(np.ascontiguousarray(t.data.view(np.int8).reshape(t.shape)[rows]),
                             xs[t.shape[1]])
        assert np.array_equal(y.cpu().numpy().astype(np.int64)[:, rows], want), t.name


def test_int8_gemm_adds_and_rejects(dev):
    rng = np.random.default_rng(51)
    w = rng.integers(-128, 128, (64, 512)).astype(np.int8)
    x = rng.integers(-128, 128, (8, 512)).astype(np.int8)
    blob = wc.encode([("u8", w, (64, 512))], tile=(16, 128), tile_order=1)
    d = wc.to_device(blob, dev)
    y0 = torch.from_numpy(oracle.gemm_i8(w, x).astype(np.int32)).to(dev)
    wc.gemm_i8_torch(blob, d, [0], [torch.from_numpy(x).to(dev)], ys=[y0])   # y += x W^T
    torch.cuda.synchronize()
    assert np.array_equal(y0.cpu().numpy().astype(np.int64), 2 * oracle.gemm_i8(w, x))
    b64 = wc.encode([("u8", w, (64, 512))], tile=(64, 128), tile_order=1)
    bf = wc.encode([("bf16", w.view(np.uint8).view(np.uint16).reshape(64, 256), (64, 256))],
                   tile=(16, 128), tile_order=1)
    for b in (b64, bf):
        with pytest.raises(wc.WcError) as e:
            _run_gemm_i8(b, dev, 0, x if b is b64 else x[:, :256])
        assert e.value.rc == -5
    with pytest.raises(wc.WcError) as e:
        _run_gemm_i8(blob, dev, 0, rng.integers(-128, 128, (65, 512)).astype(np.int8))
    assert e.value.rc == -1


# --- fp8 weights (e4m3, e5m2), bf16 x (W8A16): exact conversion, bf16 MFMA ----

FP8 = ["e4m3", "e5m2"]


def _fp8_special(w, fmt):
    """NaN patterns (e4m3), infinities and NaN (e5m2)."""
    return (w & 0x7F) == 0x7F if fmt == "e4m3" else (w & 0x7C) == 0x7C


def _fp8_codes(rng, shape, fmt):
    w = rng.integers(0, 256, shape).astype(np.uint8)
    w[_fp8_special(w, fmt)] &= 0xFB      # e4m3: exponent 15 -> mantissa 3; e5m2: exponent 30
    return w


def _fp8_value(fmt):
    return oracle.e4m3_value if fmt == "e4m3" else oracle.e5m2_value


def _check_fp8(y, w, x, fmt):
    ref, absref = oracle.gemv_fp8(w, x, fmt)
    tol = 2.0 * w.shape[1] * 2.0 ** -24 * absref + 1e-30
    bad = np.abs(y - ref) > tol
    assert not bad.any(), (np.argwhere(bad)[:5], float(np.abs(y - ref).max()))


@pytest.mark.parametrize("fmt", FP8)
@pytest.mark.parametrize("shape,tile", [((64, 256), (16, 64)), ((48, 1024), (16, 256)),
                                        ((256, 4096), (16, 4096)), ((32, 64), (16, 16))])
@pytest.mark.parametrize("m", [1, 5, 16, 17, 33, 64])
def test_fp8_gemv_matches_the_reference(dev, fmt, shape, tile, m):
    """fp8 tiles of 16 rows, converted to bf16 while decoded: y within the fp32
    summation bound of the oracle's fp64 product (every e4m3 and e5m2 value is
    a bf16 value, so the conversion adds no error)."""
    say("fp8 gemv", fmt, shape, tile, m)
    rng = np.random.default_rng(shape[1] + 11 * m + (7 if fmt == "e5m2" else 0))
    w = _fp8_codes(rng, shape, fmt)
    x = _bf16(rng.normal(0, 1.0, (m, shape[1])))
    blob = wc.encode([("fp8_" + fmt, w, shape)], tile=tile, tile_order=1)
    _check_fp8(_run_gemv(blob, dev, 0, x), w, x, fmt)


@pytest.mark.parametrize("fmt", FP8)
def test_fp8_gemv_every_code_exact(dev, fmt):
    """Every finite code of the format, picked out by one-hot rows of x: y[m][n]
    must be the code's value exactly (fp32 holds every fp8 value), which pins
    the conversion of every byte (subnormals and signed zero included), its
    byte order within the lane-group and both halves of the MFMA operand, in
    the first and the last k-block of a tile."""
    value = _fp8_value(fmt)
    K = 256
    k = np.arange(K)[None, :]
    n = np.arange(16)[:, None]
    w = ((16 * k + n) % 256).astype(np.uint8)   # columns 0..15 and 240..255 hold every code
    w[_fp8_special(w, fmt)] = 0
    cols = list(range(16)) + list(range(240, 256))
    x = np.zeros((len(cols), K), np.float32)
    for m, c in enumerate(cols):
        x[m, c] = 1.0
    blob = wc.encode([("fp8_" + fmt, w, w.shape)], tile=(16, 256), tile_order=1)
    y = _run_gemv(blob, dev, 0, _bf16(x))
    want = np.array([[value(int(w[r, c])) for r in range(16)] for c in cols])
    assert np.array_equal(y, want), np.argwhere(y != want)[:8]


@pytest.mark.parametrize("fmt", FP8)
def test_fp8_gemv_small_integers_exact(dev, fmt):
    """Small integers, exact in the format, bf16 and fp32 sums: y equals the
    integer product, which pins the conversion's byte order and both MFMA
    halves."""
    rng = np.random.default_rng(52)
    mbits, bias, top = (3, 7, 16) if fmt == "e4m3" else (2, 15, 8)
    codes = {0: 0x00}
    for v in range(1, top + 1):
        e = v.bit_length() - 1
        codes[v] = ((e + bias) << mbits) | ((v << mbits >> e) & ((1 << mbits) - 1))
        codes[-v] = 0x80 | codes[v]
    wi = rng.integers(-top, top + 1, (64, 512))
    xi = rng.integers(-40, 41, (37, 512))
    w = np.vectorize(codes.get)(wi).astype(np.uint8)
    blob = wc.encode([("fp8_" + fmt, w, w.shape)], tile=(16, 256), tile_order=1)
    y = _run_gemv(blob, dev, 0, _bf16(xi.astype(np.float32)))
    assert np.array_equal(y, (xi @ wi.T).astype(np.float64))


@pytest.mark.parametrize("fmt,cfg", [("e4m3", 6), ("e5m2", 9)])
def test_fp8_gemv_quantised_layer(dev, fmt, cfg):
    """The fp8 codes of the scaled 8B fp8 workload (per-row scales stay with the
    caller) in 16 x 512 tiles, one launch, 16 rows of x: sampled rows of y."""
    ts = [t for t in synth.config(cfg, div=4) if t.dtype == "fp8_" + fmt and len(t.shape) == 2]
    assert ts
    blob = wc.encode([(t.dtype, t.data, t.shape) for t in ts], tile=(16, 512), tile_order=1)
    d = wc.to_device(blob, dev)
    rng = np.random.default_rng(53)
    xbits = {}
    for t in ts:
        xbits.setdefault(t.shape[1], _bf16(rng.normal(0, 1.0, (16, t.shape[1]))))
    err = torch.zeros(1, dtype=torch.int32, device=dev)
    ys = wc.gemv_torch(blob, d, list(range(len(ts))), [_dev_x(xbits[t.shape[1]], dev) for t in ts],
                       err=err)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    for t, y in zip(ts, ys):
        rows = np.random.default_rng(t.shape[0]).choice(t.shape[0], 32, replace=False)
        w = np.ascontiguousarray(t.data.reshape(t.shape)[rows])
        ref, absref = oracle.gemv_fp8(w, xbits[t.shape[1]], fmt)
        tol = 2.0 * t.shape[1] * 2.0 ** -24 * absref + 1e-30
        assert (np.abs(y.cpu().numpy().astype(np.float64)[:, rows] - ref) <= tol).all(), t.name


def test_fp8_formats_in_one_call(dev):
    """e4m3 and e5m2 jobs (and a bf16 one) in one wc_gemv call: one launch per
    weight type, each job converted by its own format."""
    rng = np.random.default_rng(55)
    w4 = _fp8_codes(rng, (32, 512), "e4m3")
    w5 = _fp8_codes(rng, (48, 512), "e5m2")
    wb = _bf16(rng.normal(0, 0.02, (16, 512)))
    blob = wc.encode([("fp8_e4m3", w4, w4.shape), ("fp8_e5m2", w5, w5.shape),
                      ("bf16", wb, wb.shape)], tile=(16, 256), tile_order=1)
    x = _bf16(rng.normal(0, 1.0, (8, 512)))
    d = wc.to_device(blob, dev)
    err = torch.zeros(1, dtype=torch.int32, device=dev)
    ys = wc.gemv_torch(blob, d, [0, 1, 2], [_dev_x(x, dev)] * 3, err=err)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    _check_fp8(ys[0].cpu().numpy().astype(np.float64), w4, x, "e4m3")
    _check_fp8(ys[1].cpu().numpy().astype(np.float64), w5, x, "e5m2")
    _check(ys[2].cpu().numpy().astype(np.float64), wb, x)


@pytest.mark.parametrize("fmt", FP8)
@pytest.mark.parametrize("tiles,m", [(6144, 16), (6145, 1), (8192, 16), (8193, 16), (7000, 17)])
def test_fp8_gemv_around_the_wide_kernels_window(dev, fmt, tiles, m):
    """wc_gemv runs fp8 weights on a 16-wave kernel when the launch has one
    block of x rows (m <= 16) and its 16-row tiles overflow the 8-wave
    kernel's resident waves (6144 on a 256-CU MI355X) but fit the 16-wave
    kernel's (8192).  Per-row scaled fp8 codes of Normal(0, 1) draws, tile
    counts on both edges of that window and m = 17 (outside it): sampled rows
    of y within the fp32 summation bound of the oracle's product."""
    say("fp8 wide window", fmt, tiles, m)
    rows, cols = 16 * tiles, 512
    rng = np.random.default_rng(tiles + (3 if fmt == "e5m2" else 0))
    w, _ = synth.quant_fp8_rows(rng.standard_normal((rows, cols), dtype=np.float32), fmt)
    w[_fp8_special(w, fmt)] &= 0xFB
    blob = wc.encode([("fp8_" + fmt, w, w.shape)], tile=(16, 512), tile_order=1)
    x = _bf16(rng.normal(0, 1.0, (m, cols)))
    y = _run_gemv(blob, dev, 0, x)
    pick = np.concatenate([rng.choice(rows, 64, replace=False), [0, rows - 1]])
    _check_fp8(y[:, pick], np.ascontiguousarray(w[pick]), x, fmt)


@pytest.mark.parametrize("fmt", FP8)
def test_fp8_gemv_limits(dev, fmt):
    rng = np.random.default_rng(54)
    w = _fp8_codes(rng, (64, 512), fmt)
    b64 = wc.encode([("fp8_" + fmt, w, w.shape)], tile=(64, 256), tile_order=1)
    b16 = wc.encode([("fp8_" + fmt, w, w.shape)], tile=(16, 256), tile_order=1)
    with pytest.raises(wc.WcError) as e:                 # 64-row fp8 tiles
        _run_gemv(b64, dev, 0, _bf16(rng.normal(0, 1.0, (4, 512))))
    assert e.value.rc == -5
    with pytest.raises(wc.WcError) as e:                 # the shared path is bf16 only
        _run_gemm(b16, dev, 0, _bf16(rng.normal(0, 1.0, (65, 512))))
    assert e.value.rc == -5
    x = _bf16(rng.normal(0, 1.0, (64, 512)))
    _check_fp8(_run_gemm(b16, dev, 0, x), w, x, fmt)     # wc_gemm up to 64 rows is wc_gemv


# --- MXFP4 weights (e2m1 codes, e8m0 scale per 32), bf16 x: wc_gemv_mx --------

def _mx_pack(codes):
    """Nibble codes (rows x cols) packed two per byte, even element low."""
    return (codes[:, 0::2] | (codes[:, 1::2] << 4)).astype(np.uint8)


CODINGS = ["nibbles", "bytes"]


def _mx_encode(packed, rows, cols, tile, coding, **kw):
    """Blob of MXFP4 codes as e2m1 nibble symbols, or their packed bytes as u8
    byte symbols (tile columns in bytes)."""
    if coding == "nibbles":
        return wc.encode([("fp4_e2m1", packed, (rows, cols))], tile=tile, tile_order=1, **kw)
    return wc.encode([("u8", packed, (rows, cols // 2))], tile=(tile[0], tile[1] // 2),
                     tile_order=1, **kw)


def _run_mx(blob, dev, t, scales, x_bits, expect_err=0):
    d = wc.to_device(blob, dev)
    err = torch.zeros(1, dtype=torch.int32, device=dev)
    sc = torch.from_numpy(np.ascontiguousarray(scales, np.uint8).reshape(-1).copy()).to(dev)
    ys = wc.gemv_mx_torch(blob, d, [t], [sc], [_dev_x(x_bits, dev)], err=err)
    torch.cuda.synchronize()
    assert int(err.item()) == expect_err, wc.describe_errors(int(err.item()))
    return ys[0].cpu().numpy().astype(np.float64)


def _check_mx(y, w, sc, x):
    ref, absref = oracle.gemv_mxfp4(w, sc, x)
    tol = 2.0 * 2 * w.shape[1] * 2.0 ** -24 * absref + 1e-30
    bad = np.abs(y - ref) > tol
    assert not bad.any(), (np.argwhere(bad)[:5], float(np.abs(y - ref).max()))


@pytest.mark.parametrize("coding", CODINGS)
@pytest.mark.parametrize("varied", [False, True])
def test_mx_gemv_every_code_exact(dev, varied, coding):
    """Every e2m1 code in every position of a lane-group, picked out by one-hot
    rows of x in the first and the last MX block of a tile row: y must be the
    code's value times its block's scale exactly (fp32 holds every product),
    which pins the nibble order of the conversion, the four MFMA operands of a
    lane-group and the scale each lane-group reads."""
    rows, cols = 16, 256
    k = np.arange(cols)[None, :]
    n = np.arange(rows)[:, None]
    codes = ((n + k) % 16).astype(np.uint8)
    rng = np.random.default_rng(81)
    sc = (rng.integers(118, 137, (rows, cols // 32)) if varied
          else np.full((rows, cols // 32), 127)).astype(np.uint8)
    picks = list(range(32)) + list(range(224, 256))
    x = np.zeros((len(picks), cols), np.float32)
    for m, c in enumerate(picks):
        x[m, c] = 1.0
    blob = _mx_encode(_mx_pack(codes), rows, cols, (16, 256), coding)
    y = _run_mx(blob, dev, 0, sc, _bf16(x))
    want = np.array([[oracle.e2m1_value(int(codes[r, c])) * oracle.e8m0_value(int(sc[r, c // 32]))
                      for r in range(rows)] for c in picks])
    assert np.array_equal(y, want), np.argwhere(y != want)[:8]


@pytest.mark.parametrize("shape,tile", [((64, 512), (16, 128)), ((48, 1024), (16, 256)),
                                        ((256, 4096), (16, 4096))])
@pytest.mark.parametrize("m", [1, 5, 16, 17, 33, 64])
@pytest.mark.parametrize("coding", CODINGS)
def test_mx_gemv_matches_the_reference(dev, shape, tile, m, coding):
    """MXFP4 tiles of 16 rows, converted to bf16 with their block scales while
    decoded: y within the fp32 summation bound of the oracle's fp64 product."""
    say("mx gemv", shape, tile, m, coding)
    rng = np.random.default_rng(shape[1] + 13 * m)
    codes = rng.integers(0, 16, shape).astype(np.uint8)
    sc = rng.integers(112, 140, (shape[0], shape[1] // 32)).astype(np.uint8)
    x = _bf16(rng.normal(0, 1.0, (m, shape[1])))
    w = _mx_pack(codes)
    blob = _mx_encode(w, shape[0], shape[1], tile, coding)
    _check_mx(_run_mx(blob, dev, 0, sc, x), w, sc, x)


@pytest.mark.parametrize("coding", CODINGS)
def test_mx_gemv_small_integers_exact(dev, coding):
    """e2m1 integers (0..4, 6) at scale 1 and small integer x: every sum is an
    integer below 2^24, so y must equal the integer product exactly."""
    rng = np.random.default_rng(82)
    table = {0: 0, 1: 2, 2: 4, 3: 5, 4: 6, 6: 7}
    vals = rng.choice([0, 1, 2, 3, 4, 6, -1, -2, -3, -4, -6], (64, 512))
    codes = np.vectorize(lambda v: table[abs(v)] | (8 if v < 0 else 0))(vals).astype(np.uint8)
    xi = rng.integers(-40, 41, (37, 512))
    sc = np.full((64, 512 // 32), 127, np.uint8)
    blob = _mx_encode(_mx_pack(codes), 64, 512, (16, 256), coding)
    y = _run_mx(blob, dev, 0, sc, _bf16(xi.astype(np.float32)))
    assert np.array_equal(y, (xi @ vals.T).astype(np.float64))


@pytest.mark.parametrize("coding", CODINGS)
def test_mx_gemv_quantised_layer(dev, coding):
    """The scaled 8B MXFP4 workload as a serving step would run it: one blob
    holds the codes (16 x 512 tiles) and the scale bytes; wc_decode brings the
    scales back, one wc_gemv_mx launch multiplies all seven projections by 16
    rows of x; sampled rows of y against the oracle."""
    ts = synth.config(7, div=4)
    blocks = [t for t in ts if t.dtype == "fp4_e2m1"]
    scales = [t for t in ts if t.name.endswith(".scales")]
    assert len(blocks) == len(scales) == 7
    if coding == "nibbles":
        entries = [(t.dtype, t.data, t.shape) for t in blocks]
    else:
        entries = [("u8", t.data, (t.shape[0], t.shape[1] // 2)) for t in blocks]
    entries += [(t.dtype, t.data) for t in scales]
    blob = wc.encode(entries, tile=(16, 512 if coding == "nibbles" else 256), tile_order=1)
    d = wc.to_device(blob, dev)
    outs = wc.decode_torch(blob, d)
    dsc = outs[len(blocks):]
    rng = np.random.default_rng(83)
    xbits = {}
    for t in blocks:
        xbits.setdefault(t.shape[1], _bf16(rng.normal(0, 1.0, (16, t.shape[1]))))
    err = torch.zeros(1, dtype=torch.int32, device=dev)
    ys = wc.gemv_mx_torch(blob, d, list(range(len(blocks))), dsc,
                          [_dev_x(xbits[t.shape[1]], dev) for t in blocks], err=err)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    for t, s, y in zip(blocks, scales, ys):
        rows = np.random.default_rng(t.shape[0]).choice(t.shape[0], 32, replace=False)
        w = np.ascontiguousarray(t.data.reshape(t.shape[0], -1)[rows])
        sc = np.ascontiguousarray(s.data.reshape(t.shape[0], -1)[rows])
        ref, absref = oracle.gemv_mxfp4(w, sc, xbits[t.shape[1]])
        tol = 2.0 * t.shape[1] * 2.0 ** -24 * absref + 1e-30
        assert (np.abs(y.cpu().numpy().astype(np.float64)[:, rows] - ref) <= tol).all(), t.name


@pytest.mark.parametrize("tiles,m", [(6144, 8), (6145, 1), (8192, 8), (8193, 8), (7000, 9)])
def test_mx_gemv_bytes_around_the_wide_kernels_window(dev, tiles, m):
    """MXFP4 codes coded as bytes run on a 16-wave kernel when the launch has
    up to 8 rows of x and its 16-row tiles overflow the 8-wave
    kernel's resident waves (6144 on a 256-CU MI355X) but fit the 16-wave
    kernel's (8192).  Tile counts on both edges of that window and m = 9
    (outside it): sampled rows of y within the fp32 summation bound of the
    oracle's product."""
    say("mx bytes wide window", tiles, m)
    rows, cols = 16 * tiles, 512
    rng = np.random.default_rng(tiles + 5)
    w = _mx_pack(rng.integers(0, 16, (rows, cols)).astype(np.uint8))
    sc = rng.integers(112, 140, (rows, cols // 32)).astype(np.uint8)
    x = _bf16(rng.normal(0, 1.0, (m, cols)))
    y = _run_mx(_mx_encode(w, rows, cols, (16, 512), "bytes"), dev, 0, sc, x)
    pick = np.concatenate([rng.choice(rows, 64, replace=False), [0, rows - 1]])
    _check_mx(y[:, pick], np.ascontiguousarray(w[pick]), np.ascontiguousarray(sc[pick]), x)


def test_mx_gemv_limits(dev):
    rng = np.random.default_rng(84)
    codes = rng.integers(0, 16, (64, 512)).astype(np.uint8)
    w = _mx_pack(codes)
    sc = np.full((64, 16), 127, np.uint8)
    x = _bf16(rng.normal(0, 1.0, (4, 512)))
    for tile in [(64, 256), (16, 64), (32, 128)]:        # not 16 rows x 128k columns
        blob = wc.encode([("fp4_e2m1", w, codes.shape)], tile=tile, tile_order=1)
        with pytest.raises(wc.WcError) as e:
            _run_mx(blob, dev, 0, sc, x)
        assert e.value.rc == -5, tile
    blob = wc.encode([("u8", w, (64, 256))], tile=(16, 32), tile_order=1)
    with pytest.raises(wc.WcError) as e:                 # byte-coded tile of 64 codes
        _run_mx(blob, dev, 0, sc, x)
    assert e.value.rc == -5
    blob = wc.encode([("u4", w, codes.shape)], tile=(16, 128), tile_order=1)
    with pytest.raises(wc.WcError) as e:                 # int4 codes are not e2m1
        _run_mx(blob, dev, 0, sc, x)
    assert e.value.rc == -5
    blob = wc.encode([("fp4_e2m1", w, codes.shape)], tile=(16, 128), tile_order=1)
    d = wc.to_device(blob, dev)
    y = torch.zeros((4, 64), dtype=torch.float32, device=dev)
    with pytest.raises(wc.WcError) as e:                 # no scales
        wc.gemv_mx(blob, d.data_ptr(), [0], [0], [_dev_x(x, dev).data_ptr()], 4, [y.data_ptr()])
    assert e.value.rc == -1
    with pytest.raises(wc.WcError) as e:                 # 65 rows of x
        wc.gemv_mx(blob, d.data_ptr(), [0], [1], [_dev_x(x, dev).data_ptr()], 65, [y.data_ptr()])
    assert e.value.rc == -1


# --- group-quantised int4 weights (codes as bytes), bf16 x: wc_gemv_w4 ---------

def _w4_pack(codes):
    return (codes[:, 0::2] | (codes[:, 1::2] << 4)).astype(np.uint8)


def _run_w4(blob, dev, scales, zeros, x_bits, expect_err=0):
    d = wc.to_device(blob, dev)
    err = torch.zeros(1, dtype=torch.int32, device=dev)
    sc = torch.from_numpy(np.ascontiguousarray(scales, np.uint16).view(np.int16).reshape(-1).copy()).to(dev)
    zs = None if zeros is None else [torch.from_numpy(np.ascontiguousarray(zeros, np.uint8).reshape(-1).copy()).to(dev)]
    ys = wc.gemv_w4_torch(blob, d, [0], [sc], zs, [_dev_x(x_bits, dev)], err=err)
    torch.cuda.synchronize()
    assert int(err.item()) == expect_err, wc.describe_errors(int(err.item()))
    return ys[0].cpu().numpy().astype(np.float64)


def _w4_tolerance(w, sc, zeros, x_bits, absref):
    """fp32 error bound of y: per group, sums of 128 products with x of
    (16 + t) and of ones, the correction (16 + z or 24) times the second, the
    scale, and the fp32 accumulation over groups and tiles (u = 2^-24):
    u (10^4 sum_g |s_g| sum_{k in g} |x_k| + (K/128 + 64) sum |x w|)."""
    K = 2 * w.shape[1]
    xv = (np.asarray(x_bits, np.uint32) << 16).view(np.float32).astype(np.float64)
    gx = np.abs(xv).reshape(xv.shape[0], K // 128, 128).sum(axis=2)            # M x G
    s = np.abs(np.ascontiguousarray(sc, np.uint16).view(np.float16).astype(np.float64))  # N x G
    return 2.0 ** -24 * (1e4 * (gx @ s.T) + (K / 128 + 64) * absref) + 1e-30


def _w4_encode(w, rows, cols, tile_bytes, coding):
    """Blob of int4 codes as u8 byte symbols (tile columns in bytes) or u4 nibbles."""
    if coding == "bytes":
        return wc.encode([("u8", w, (rows, cols // 2))], tile=(16, tile_bytes), tile_order=1)
    return wc.encode([("u4", w, (rows, cols))], tile=(16, 2 * tile_bytes), tile_order=1)


@pytest.mark.parametrize("coding", CODINGS)
@pytest.mark.parametrize("with_zeros", [False, True])
def test_w4_gemv_every_code_exact(dev, with_zeros, coding):
    """Every code in every position of a lane-group and in the first and last
    group of a tile row, picked by one-hot x rows at scale 1: y must be q - z
    (or the signed code) exactly, which pins the nibble order, the +16 / +8
    offsets, the sums of x through the ones operand and the group of each
    wave row."""
    rows, cols = 16, 512
    k = np.arange(cols)[None, :]
    n = np.arange(rows)[:, None]
    codes = ((n + k) % 16).astype(np.uint8)
    rng = np.random.default_rng(91)
    zeros = rng.integers(0, 16, (rows, cols // 128)).astype(np.uint8) if with_zeros else None
    sc = np.full((rows, cols // 128), 0x3C00, np.uint16)
    picks = list(range(32)) + list(range(480, 512))
    x = np.zeros((len(picks), cols), np.float32)
    for m, c in enumerate(picks):
        x[m, c] = 1.0
    w = _w4_pack(codes)
    blob = _w4_encode(w, rows, cols, 256, coding)
    y = _run_w4(blob, dev, sc, zeros, _bf16(x))
    want = np.array([[(int(codes[r, c]) - int(zeros[r, c // 128])) if with_zeros
                      else (int(codes[r, c]) ^ 8) - 8 for r in range(rows)] for c in picks],
                    np.float64)
    assert np.array_equal(y, want), np.argwhere(y != want)[:8]


@pytest.mark.parametrize("with_zeros", [False, True])
@pytest.mark.parametrize("shape,tile", [((64, 512), (16, 64)), ((48, 1024), (16, 128)),
                                        ((256, 4096), (16, 2048))])
@pytest.mark.parametrize("m", [1, 5, 16, 17, 33, 64])
@pytest.mark.parametrize("coding", CODINGS)
def test_w4_gemv_matches_the_reference(dev, with_zeros, shape, tile, m, coding):
    """Random codes, fp16 scales and zero points: y within the derived fp32
    bound of the oracle's fp64 product."""
    say("w4 gemv", with_zeros, shape, tile, m, coding)
    rng = np.random.default_rng(shape[1] + 17 * m + with_zeros)
    codes = rng.integers(0, 16, shape).astype(np.uint8)
    sc = rng.uniform(0.002, 0.05, (shape[0], shape[1] // 128)).astype(np.float16).view(np.uint16)
    zeros = rng.integers(0, 16, (shape[0], shape[1] // 128)).astype(np.uint8) if with_zeros else None
    x = _bf16(rng.normal(0, 1.0, (m, shape[1])))
    w = _w4_pack(codes)
    blob = _w4_encode(w, shape[0], shape[1], tile[1], coding)
    y = _run_w4(blob, dev, sc, zeros, x)
    ref, absref = oracle.gemv_int4(w, sc, zeros, x)
    tol = _w4_tolerance(w, sc, zeros, x, absref)
    bad = np.abs(y - ref) > tol
    assert not bad.any(), (np.argwhere(bad)[:5], float(np.abs(y - ref).max()))


def test_w4_gemv_small_integers_exact(dev):
    """Scale 1, zero points, small integer x: every partial sum is an integer
    below 2^24, so y must equal the oracle's integer product exactly."""
    rng = np.random.default_rng(92)
    codes = rng.integers(0, 16, (64, 1024)).astype(np.uint8)
    zeros = rng.integers(0, 16, (64, 8)).astype(np.uint8)
    sc = np.full((64, 8), 0x3C00, np.uint16)
    xi = rng.integers(-40, 41, (37, 1024))
    w = _w4_pack(codes)
    blob = wc.encode([("u8", w, (64, 512))], tile=(16, 256), tile_order=1)
    y = _run_w4(blob, dev, sc, zeros, _bf16(xi.astype(np.float32)))
    ref, _ = oracle.gemv_int4(w, sc, zeros, _bf16(xi.astype(np.float32)))
    assert np.array_equal(y, ref)


@pytest.mark.parametrize("coding", CODINGS)
@pytest.mark.parametrize("cfg", [3, 8])
def test_w4_gemv_quantised_layer(dev, cfg, coding):
    """The scaled 8B int4 (two's-complement codes) and AWQ-style (zero points)
    workloads as a serving step: one blob holds the codes as bytes (16 x 256-byte
    tiles), the fp16 scales and the packed zero points; wc_decode brings the
    scales and zeros back, torch unpacks the zero nibbles to bytes, one
    wc_gemv_w4 launch multiplies all seven projections by 16 rows of x; sampled
    rows of y against the oracle."""
    ts = synth.config(cfg, div=4)
    codes = [t for t in ts if t.name.endswith(".qweight")]
    scales = [t for t in ts if t.name.endswith(".scales")]
    zeros = [t for t in ts if t.name.endswith(".qzeros")]
    assert len(codes) == len(scales) == 7 and len(zeros) in (0, 7)
    if coding == "bytes":
        entries = [("u8", t.data, (t.shape[0], t.shape[1] // 2)) for t in codes]
    else:
        entries = [(t.dtype, t.data, t.shape) for t in codes]
    entries += [(t.dtype, t.data) for t in scales + zeros]
    blob = wc.encode(entries, tile=(16, 256 if coding == "bytes" else 512), tile_order=1)
    d = wc.to_device(blob, dev)
    outs = wc.decode_torch(blob, d)
    dsc = outs[7:14]
    dz = None
    if zeros:
        dz = [torch.stack([o & 15, o >> 4], dim=1).reshape(-1).contiguous() for o in outs[14:21]]
    rng = np.random.default_rng(93)
    xbits = {}
    for t in codes:
        xbits.setdefault(t.shape[1], _bf16(rng.normal(0, 1.0, (16, t.shape[1]))))
    err = torch.zeros(1, dtype=torch.int32, device=dev)
    ys = wc.gemv_w4_torch(blob, d, list(range(7)), dsc, dz,
                          [_dev_x(xbits[t.shape[1]], dev) for t in codes], err=err)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    for j, (t, s, y) in enumerate(zip(codes, scales, ys)):
        rows = np.random.default_rng(t.shape[0]).choice(t.shape[0], 32, replace=False)
        w = np.ascontiguousarray(t.data.reshape(t.shape[0], -1)[rows])
        sc = np.ascontiguousarray(s.data.reshape(t.shape[0], -1)[rows]).view(np.uint16)
        z = None
        if zeros:
            zp = zeros[j].data.reshape(t.shape[0], -1)
            z = np.ascontiguousarray(np.stack([zp & 15, zp >> 4], axis=2).reshape(t.shape[0], -1)[rows])
        ref, absref = oracle.gemv_int4(w, sc, z, xbits[t.shape[1]])
        tol = _w4_tolerance(w, sc, z, xbits[t.shape[1]], absref)
        assert (np.abs(y.cpu().numpy().astype(np.float64)[:, rows] - ref) <= tol).all(), t.name


@pytest.mark.parametrize("tiles,m", [(6144, 8), (6145, 1), (8192, 8), (8193, 8), (7000, 9)])
def test_w4_gemv_bytes_around_the_wide_kernels_window(dev, tiles, m):
    """int4 codes coded as bytes run on a 16-wave kernel when the launch has
    up to 8 rows of x and its 16-row tiles overflow the 8-wave
    kernel's resident waves (6144 on a 256-CU MI355X) but fit the 16-wave
    kernel's (8192).  Tile counts on both edges of that window and m = 9
    (outside it), with zero points on odd tile counts: sampled rows of y
    within the derived bound of the oracle's product."""
    say("w4 bytes wide window", tiles, m)
    rows, cols = 16 * tiles, 512
    rng = np.random.default_rng(tiles + 9)
    w = _w4_pack(rng.integers(0, 16, (rows, cols)).astype(np.uint8))
    sc = rng.uniform(0.002, 0.05, (rows, cols // 128)).astype(np.float16).view(np.uint16)
    zeros = rng.integers(0, 16, (rows, cols // 128)).astype(np.uint8) if tiles % 2 else None
    x = _bf16(rng.normal(0, 1.0, (m, cols)))
    y = _run_w4(_w4_encode(w, rows, cols, 256, "bytes"), dev, sc, zeros, x)
    pick = np.concatenate([rng.choice(rows, 64, replace=False), [0, rows - 1]])
    wp, sp = np.ascontiguousarray(w[pick]), np.ascontiguousarray(sc[pick])
    zp = None if zeros is None else np.ascontiguousarray(zeros[pick])
    ref, absref = oracle.gemv_int4(wp, sp, zp, x)
    tol = _w4_tolerance(wp, sp, zp, x, absref)
    assert (np.abs(y[:, pick] - ref) <= tol).all()


def test_w4_gemv_limits(dev):
    rng = np.random.default_rng(94)
    codes = rng.integers(0, 16, (64, 512)).astype(np.uint8)
    w = _w4_pack(codes)
    sc = np.full((64, 4), 0x3C00, np.uint16)
    x = _bf16(rng.normal(0, 1.0, (4, 512)))
    for entry, tile in [(("u8", w, (64, 256)), (16, 32)),     # 64 codes per tile row
                        (("u8", w, (64, 256)), (64, 128)),    # 64-row tiles
                        (("u4", w, (64, 512)), (16, 64))]:    # 64 nibbles wide
        blob = wc.encode([entry], tile=tile, tile_order=1)
        with pytest.raises(wc.WcError) as e:
            _run_w4(blob, dev, sc, None, x)
        assert e.value.rc == -5, tile
    blob = wc.encode([("u8", w, (64, 256))], tile=(16, 128), tile_order=1)
    d = wc.to_device(blob, dev)
    y = torch.zeros((4, 64), dtype=torch.float32, device=dev)
    with pytest.raises(wc.WcError) as e:                 # scales not 2-byte aligned
        wc.gemv_w4(blob, d.data_ptr(), [0], [17], None, [_dev_x(x, dev).data_ptr()], 4,
                   [y.data_ptr()])
    assert e.value.rc == -1
