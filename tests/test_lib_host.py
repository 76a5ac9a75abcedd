"""CPU tests of libwc's host half: exports, analysis, encoder, blob validation.

No GPU call is made here.  The library's encoder is separate code from the
oracle's; both follow the same format readings, so their blobs must be
byte-identical, and the library's statistics must equal the oracle's.
"""
import ctypes as C
import math
import os
import re
import struct
import subprocess

import numpy as np
import pytest

import oracle
from paper_2606_15789_amd import synth, wc

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    text = open(os.path.join(ROOT, "include", "wc.h")).read()
    return sorted(set(re.findall(r"^\s*(?:wc_status|void|int32_t)\s+(wc_\w+)\s*\(", text, re.M)))


def test_library_exports_every_declared_symbol():
    names = declared_functions()
    assert set(names) == set(wc.EXPORTS)
    lib = wc.lib()
    for n in names:
        assert hasattr(lib, n), n
    out = subprocess.run(["nm", "-D", "--defined-only", wc.library_path()], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r"\bT (wc_\w+)", out))
    assert set(names) <= exported
    assert lib.wc_version() == 12


@pytest.mark.parametrize("cfg,div", [(1, 4), (2, 8), (3, 8), (4, 8), (5, 16), (6, 8), (7, 8),
                                     (8, 8), (9, 8)])
@pytest.mark.parametrize("lanes", [64, 32])
def test_blobs_identical_to_oracle(cfg, div, lanes):
    ts = synth.config(cfg, div=div)
    pairs = [(t.dtype, t.data) for t in ts]
    for cb in (16384, 65536):
        b = wc.encode(pairs, chunk_bytes=cb, lanes=lanes, threads=4)
        assert b.tobytes() == oracle.encode(pairs, chunk_bytes=cb, lanes=lanes)
        assert sum(b.breakdown.values()) == b.size
        assert b.out_bytes == [t.nbytes for t in ts]


def test_blob_identical_on_edge_sizes_and_patterns():
    rng = np.random.default_rng(2)
    allw = rng.permutation(np.arange(65536, dtype=np.uint32)).astype(np.uint16)
    pairs = [("bf16", allw), ("fp16", allw[:1001]), ("u8", np.zeros(0, np.uint8)),
             ("u4", rng.integers(0, 256, 777).astype(np.uint8)), ("u8", np.full(5, 9, np.uint8)),
             ("bf16", allw[:1]), ("fp8_e5m2", rng.integers(0, 256, 3001).astype(np.uint8)),
             ("fp4_e2m1", rng.integers(0, 256, 513).astype(np.uint8)),
             ("fp8_e4m3", np.zeros(0, np.uint8))]
    for lanes in (1, 7, 64):
        for cb in (256, 1024):
            assert wc.encode(pairs, chunk_bytes=cb, lanes=lanes).tobytes() == \
                oracle.encode(pairs, chunk_bytes=cb, lanes=lanes)


def test_encoder_is_thread_count_invariant():
    pairs = [(t.dtype, t.data) for t in synth.config(2, div=8)]
    ref = wc.encode(pairs, threads=1).tobytes()
    for th in (2, 3, 8):
        assert wc.encode(pairs, threads=th).tobytes() == ref


@pytest.mark.parametrize("cfg", [1, 3, 4, 6, 7])
def test_analyze_matches_oracle(cfg):
    for t in synth.config(cfg, div=8):
        a, o = wc.analyze(t.dtype, t.data), oracle.analyze(t.dtype, t.data)
        assert a["n_fields"] == o["n_fields"] and a["count"] == o["count"]
        for f in range(a["n_fields"]):
            assert np.array_equal(a["hist"][f], o["hist"][f])
            assert a["H"][f] == pytest.approx(o["H"][f], rel=1e-12)
        assert a["bound_bytes"] == pytest.approx(o["bound_bytes"], rel=1e-12)
        if t.dtype in ("bf16", "fp16"):
            assert a["H_joint16"] == pytest.approx(o["H_joint16"], rel=1e-12)
        else:
            assert math.isnan(a["H_joint16"])


def test_open_accepts_oracle_blob_and_rejects_corruption():
    pairs = [(t.dtype, t.data) for t in synth.config(3, div=16)]
    ob = oracle.encode(pairs, chunk_bytes=16384)
    b = wc.open_blob(ob)
    assert b.tobytes() == ob and b.n_tensors == len(pairs)
    bad_cases = []
    for pos, val in [(0, 0x00), (4, 0x07), (64 + 43, 11), (64 + 40, 0)]:
        x = bytearray(ob)
        x[pos] = val
        bad_cases.append(bytes(x))
    x = bytearray(ob)                        # frequency table no longer sums to 4096
    foff = struct.unpack_from("<Q", ob, 64 + 48)[0]
    struct.pack_into("<H", x, foff, struct.unpack_from("<H", ob, foff)[0] + 1)
    bad_cases.append(bytes(x))
    x = bytearray(ob)                        # index entry out of order
    idx = struct.unpack_from("<Q", ob, 32)[0]
    struct.pack_into("<I", x, idx + 4, 0)
    bad_cases.append(bytes(x))
    bad_cases.append(ob[:-16])               # truncated
    for bad in bad_cases:
        with pytest.raises(wc.WcError) as e:
            wc.open_blob(bad)
        assert e.value.rc == -1


def test_encode_rejects_bad_parameters():
    d = np.zeros(100, np.uint16)
    for kw in [dict(chunk_bytes=100), dict(chunk_bytes=1 << 21), dict(lanes=0), dict(lanes=65)]:
        with pytest.raises(wc.WcError):
            wc.encode([("bf16", d)], **kw)
    with pytest.raises(wc.WcError):
        wc.encode([("bf16", np.zeros(3, np.uint8))])   # odd byte count for a 16-bit format


def test_decode_rejects_before_any_launch():
    for lanes in (1, 16, 48, 63):
        b = wc.encode([("bf16", np.zeros(1000, np.uint16))], lanes=lanes)
        with pytest.raises(wc.WcError) as e:      # lane count the GPU path does not take
            wc.decode(b, 1, [1])
        assert e.value.rc == -5
    b = wc.encode([("bf16", np.zeros(1000, np.uint16))])
    with pytest.raises(wc.WcError) as e:          # tensor count mismatch
        wc.decode(b, 1, [1, 1])
    assert e.value.rc == -1
    with pytest.raises(wc.WcError):
        wc.decode(b, 0, [1])                      # no device blob


def test_stream_rejects_before_any_launch():
    """wc_stream checks sizes and alignment on the host (fake device addresses,
    never touched)."""
    for args in ((0, 32, 16, 64),             # no source
                 (16, 32, 0, 64),             # no destination
                 (16, 0, 16, 64),             # nothing to read
                 (16, 24, 16, 64),            # source not whole 16-byte units
                 (16, 32, 16, 40),            # destination not whole units
                 (8, 32, 16, 64),             # source misaligned
                 (16, 32, 24, 64),            # destination misaligned
                 (16, 128, 16, 64),           # more read than written
                 (16, 32, 16, 1 << 36)):      # destination of 2^32 units
        with pytest.raises(wc.WcError) as e:
            wc.stream_bytes(*args)
        assert e.value.rc == -1, args


@pytest.mark.parametrize("tile", [(32, 128), (64, 256), (128, 256)])
@pytest.mark.parametrize("codebook", ["tensor", "layer"])
@pytest.mark.parametrize("lanes", [64, 32])
@pytest.mark.parametrize("order", [0, 1])
def test_tiled_blobs_identical_to_oracle(tile, codebook, lanes, order):
    ts = synth.config(2, div=8) + synth.config(3, div=8)
    pairs = [(t.dtype, t.data, t.shape if len(t.shape) == 2 else None) for t in ts]
    a = wc.encode(pairs, chunk_bytes=16384, lanes=lanes, tile=tile, codebook=codebook,
                  tile_order=order)
    b = oracle.encode(pairs, chunk_bytes=16384, lanes=lanes, tile=tile, codebook=codebook,
                      tile_order=order)
    assert a.tobytes() == b
    info = oracle.tensor_info(b)
    assert any(i["tile"] == tile for i in info)            # some tensors were tiled


def test_open_rejects_inconsistent_tile_fields():
    d = np.arange(64 * 256, dtype=np.uint16).reshape(64, 256)
    raw = bytearray(oracle.encode([("bf16", d, (64, 256))], tile=(32, 128)))
    assert wc.open_blob(bytes(raw)).n_chunks == 4
    for off, val in ((64 + 80, 33), (64 + 84, 96), (64 + 72, 255)):   # rows, tile_c, cols
        bad = bytearray(raw)
        struct.pack_into("<I", bad, off, val)
        with pytest.raises(wc.WcError):
            wc.open_blob(bytes(bad))


def test_gemv_rejects_before_any_launch():
    w = (np.random.default_rng(3).normal(0, 0.02, (128, 512)).astype(np.float32)
         .view(np.uint32) >> 16).astype(np.uint16)
    good = wc.encode([("bf16", w, (128, 512))], tile=(64, 256), tile_order=1)
    rows = wc.encode([("bf16", w, (128, 512))], tile=(64, 256), tile_order=0)
    flat = wc.encode([("bf16", w, (128, 512))])
    for m in (0, 65):
        with pytest.raises(wc.WcError) as e:
            wc.gemv(good, 16, [0], [16], m, [16])
        assert e.value.rc == -1
    for m in (0, 4097):
        with pytest.raises(wc.WcError) as e:
            wc.gemm(good, 16, [0], [16], m, [16], 256, 1 << 20)
        assert e.value.rc == -1
    tile16 = wc.encode([("bf16", w, (128, 512))], tile=(16, 256), tile_order=1)
    ragged = wc.encode([("bf16", w[:100], (100, 512))], tile=(64, 256), tile_order=1)
    for b in (tile16, ragged):                    # past 64 rows: full 64-row tiles only
        with pytest.raises(wc.WcError) as e:
            wc.gemm(b, 16, [0], [16], 65, [16], 256, 1 << 20)
        assert e.value.rc == -5
    need = wc.gemm_workspace_bytes(good, [0], [16], 65)
    for ws, size in ((0, need), (256, need - 1), (16, need)):   # none, too small, misaligned
        with pytest.raises(wc.WcError) as e:
            wc.gemm(good, 16, [0], [16], 65, [16], ws, size)
        assert e.value.rc == -1

    narrow = wc.encode([("bf16", w, (128, 512))], tile=(64, 8), tile_order=1)
    with pytest.raises(wc.WcError) as e:          # 64-row tiles past 5 rows pair k-blocks
        wc.gemv(narrow, 16, [0], [16], 6, [16])
    assert e.value.rc == -5
    for args in (([0], [8], [16]),            # x not 16-byte aligned
                 ([1], [16], [16]),           # no such tensor
                 ([0], [16], [0]),            # no y
                 ([], [], []),                # no jobs
                 ([0] * 33, [16] * 33, [16] * 33)):   # more than one launch holds
        with pytest.raises(wc.WcError) as e:
            wc.gemv(good, 16, args[0], args[1], 1, args[2])
        assert e.value.rc == -1, args
    for b in (rows, flat):                      # not the column-block layout
        with pytest.raises(wc.WcError) as e:
            wc.gemv(b, 16, [0], [16], 1, [16])
        assert e.value.rc == -5


def test_gemv_mx_rejects_before_any_launch():
    """wc_gemv_mx validates every argument and tensor on the host and returns
    before any HIP call; the fake device addresses are never touched."""
    codes = np.random.default_rng(4).integers(0, 16, (64, 512)).astype(np.uint8)
    w = (codes[:, 0::2] | (codes[:, 1::2] << 4)).astype(np.uint8)
    nib = wc.encode([("fp4_e2m1", w, (64, 512))], tile=(16, 256), tile_order=1)
    for m in (0, 65):
        with pytest.raises(wc.WcError) as e:
            wc.gemv_mx(nib, 16, [0], [16], [16], m, [16])
        assert e.value.rc == -1
    for args in (([0], [0], [16], [16]),           # no scales
                 ([0], [16], [8], [16]),           # x not 16-byte aligned
                 ([1], [16], [16], [16]),          # no such tensor
                 ([0], [16], [16], [0]),           # no y
                 ([], [], [], []),                 # no jobs
                 ([0] * 33, [16] * 33, [16] * 33, [16] * 33)):
        with pytest.raises(wc.WcError) as e:
            wc.gemv_mx(nib, 16, args[0], args[1], args[2], 1, args[3])
        assert e.value.rc == -1, args
    unsupported = [
        wc.encode([("fp4_e2m1", w, (64, 512))], tile=(64, 256), tile_order=1),   # 64-row tiles
        wc.encode([("fp4_e2m1", w, (64, 512))], tile=(16, 64), tile_order=1),    # 64 codes wide
        wc.encode([("fp4_e2m1", w, (64, 512))], tile=(16, 256), tile_order=0),   # row-major tiles
        wc.encode([("fp4_e2m1", w, (64, 512))]),                                 # byte runs
        wc.encode([("u4", w, (64, 512))], tile=(16, 256), tile_order=1),         # int4 codes
        wc.encode([("u8", w, (64, 256))], tile=(16, 32), tile_order=1),          # 64 codes as bytes
        wc.encode([("fp4_e2m1", w, (64, 512))], lanes=32, tile=(16, 256), tile_order=1),
    ]
    for b in unsupported:
        with pytest.raises(wc.WcError) as e:
            wc.gemv_mx(b, 16, [0], [16], [16], 1, [16])
        assert e.value.rc == -5


def test_gemv_w4_rejects_before_any_launch():
    """wc_gemv_w4 validates every argument and tensor on the host and returns
    before any HIP call; the fake device addresses are never touched."""
    codes = np.random.default_rng(5).integers(0, 16, (64, 512)).astype(np.uint8)
    w = (codes[:, 0::2] | (codes[:, 1::2] << 4)).astype(np.uint8)
    good = wc.encode([("u8", w, (64, 256))], tile=(16, 128), tile_order=1)
    for m in (0, 65):
        with pytest.raises(wc.WcError) as e:
            wc.gemv_w4(good, 16, [0], [16], None, [16], m, [16])
        assert e.value.rc == -1
    for args in (([0], [0], [16], [16]),           # no scales
                 ([0], [17], [16], [16]),          # scales not 2-byte aligned
                 ([0], [16], [8], [16]),           # x not 16-byte aligned
                 ([1], [16], [16], [16]),          # no such tensor
                 ([0], [16], [16], [0]),           # no y
                 ([], [], [], [])):                # no jobs
        with pytest.raises(wc.WcError) as e:
            wc.gemv_w4(good, 16, args[0], args[1], None, args[2], 1, args[3])
        assert e.value.rc == -1, args
    unsupported = [
        wc.encode([("u8", w, (64, 256))], tile=(64, 128), tile_order=1),   # 64-row tiles
        wc.encode([("u8", w, (64, 256))], tile=(16, 32), tile_order=1),    # 64 codes wide
        wc.encode([("u8", w, (64, 256))], tile=(16, 128), tile_order=0),   # row-major tiles
        wc.encode([("u8", w, (64, 256))]),                                 # byte runs
        wc.encode([("u4", w, (64, 512))], tile=(16, 64), tile_order=1),    # 64 nibbles wide
        wc.encode([("fp4_e2m1", w, (64, 512))], tile=(16, 256), tile_order=1),  # e2m1 codes
        wc.encode([("u8", w, (64, 256))], lanes=32, tile=(16, 128), tile_order=1),
    ]
    for b in unsupported:
        with pytest.raises(wc.WcError) as e:
            wc.gemv_w4(b, 16, [0], [16], None, [16], 1, [16])
        assert e.value.rc == -5


def test_fused_torch_wrappers_check_tensor_sizes():
    """gemv_w4_torch and gemv_mx_torch size every scale, zero-point and x
    tensor against the weights' shape before any launch: the kernels size
    their reads from the blob, so a packed zero-point tensor (two groups a
    byte), a short scale tensor or an x of the wrong width would otherwise be
    read past its end.  CPU tensors: the checks run before any device call."""
    import torch
    N, K = 64, 512
    codes = np.random.default_rng(6).integers(0, 16, (N, K)).astype(np.uint8)
    w = (codes[:, 0::2] | (codes[:, 1::2] << 4)).astype(np.uint8)
    for blob in (wc.encode([("u8", w, (N, K // 2))], tile=(16, 128), tile_order=1),
                 wc.encode([("u4", w, (N, K))], tile=(16, 256), tile_order=1)):
        assert wc._codes_shape(blob, 0) == (N, K)
        x = torch.zeros((2, K), dtype=torch.bfloat16)
        sc = torch.zeros(N * K // 128, dtype=torch.float16)
        z = torch.zeros(N * K // 128, dtype=torch.uint8)
        bad = [
            dict(zeros=[torch.zeros(N * K // 256, dtype=torch.uint8)]),   # packed zero points
            dict(zeros=[z.to(torch.int32)]),                               # not one byte a group
            dict(scales=[sc[:-1]]),                                        # one scale short
            dict(xs=[x[:, :K - 128].contiguous()]),                        # x narrower than K
            dict(xs=[torch.zeros((2, K), dtype=torch.float32)]),           # x not bf16
            dict(xs=[x, x]),                                               # two x for one job
        ]
        for b in bad:
            kw = dict(scales=[sc], zeros=[z], xs=[x])
            kw.update(b)
            with pytest.raises(ValueError):
                wc.gemv_w4_torch(blob, None, [0], kw["scales"], kw["zeros"], kw["xs"])
    mx = wc.encode([("fp4_e2m1", w, (N, K))], tile=(16, 256), tile_order=1)
    x = torch.zeros((2, K), dtype=torch.bfloat16)
    sc = torch.zeros(N * K // 32, dtype=torch.uint8)
    for scales, xs in (([sc[:-1]], [x]),                     # one scale short
                       ([sc.to(torch.int16)], [x]),          # scales not bytes
                       ([sc], [x[:, :256].contiguous()]),    # x narrower than K
                       ([sc], [x, x])):                      # two x for one job
        with pytest.raises(ValueError):
            wc.gemv_mx_torch(mx, None, [0], scales, xs)


def test_gemm_workspace_bytes():
    """One packed x per distinct (pointer, K): rows rounded up to 32, bf16,
    each slot rounded up to 256 bytes; nothing below 65 rows."""
    w = (np.random.default_rng(5).normal(0, 0.02, (128, 512)).astype(np.float32)
         .view(np.uint32) >> 16).astype(np.uint16)
    w2 = np.ascontiguousarray(w[:, :496])
    b = wc.encode([("bf16", w, (128, 512)), ("bf16", w2, (128, 496))], tile=(64, 16),
                  tile_order=1)
    assert wc.gemm_workspace_bytes(b, [0], [16], 64) == 0
    assert wc.gemm_workspace_bytes(b, [0], [16], 65) == 96 * 512 * 2
    assert wc.gemm_workspace_bytes(b, [0, 0], [16, 16], 100) == 128 * 512 * 2
    assert wc.gemm_workspace_bytes(b, [0, 0], [16, 32], 100) == 2 * 128 * 512 * 2
    assert wc.gemm_workspace_bytes(b, [0, 1], [16, 16], 33 + 64) == (
        128 * 512 * 2 + ((128 * 496 * 2 + 255) // 256) * 256)
    with pytest.raises(wc.WcError):
        wc.gemm_workspace_bytes(b, [2], [16], 100)


def _pad16(x):
    return (x + 15) // 16 * 16


@pytest.mark.parametrize("lanes,cb,tile", [(64, 65536, (0, 0)), (32, 16384, (0, 0)),
                                           (7, 256, (0, 0)), (64, 16384, (32, 128))])
def test_device_encoder_bounds(lanes, cb, tile):
    """wc_encode_device_bounds (host only): the capacity is the blob that every
    coded symbol emitting a word would give, so any real blob fits in it."""
    ts = synth.config(2, div=8) + synth.config(3, div=8)
    entries = [(t.dtype, t.data, t.shape if len(t.shape) == 2 else None) for t in ts]
    cap, ws = wc.encode_device_bounds([(d, a.nbytes, s) for d, a, s in entries], chunk_bytes=cb,
                                      lanes=lanes, tile=tile)
    b = wc.encode(entries, chunk_bytes=cb, lanes=lanes, tile=tile, threads=4)
    assert b.size <= cap
    worst = 0
    W = {"bf16": 8, "fp16": 8, "u8": 16, "fp8_e4m3": 16, "fp8_e5m2": 16, "u4": 32,
         "fp4_e2m1": 32}
    for info, (dt, a, s) in zip(oracle.tensor_info(b.tobytes()), entries):
        n_sym = a.nbytes * W[dt] // 16          # a lane-group of W symbols is 16 bytes
        per = info["chunk_bytes"] * W[dt] // 16
        for c in range(info["n_chunks"]):
            n_c = min(per, n_sym - c * per)
            A = min(lanes, -(-n_c // W[dt]))
            worst += 16 + _pad16(4 * A) + _pad16(2 * n_c)
    assert cap == b.breakdown["meta_bytes"] + worst + b.breakdown["raw_bytes"]
    assert ws >= worst


def test_device_encoder_bounds_rejects_bad_arguments():
    e = [("u8", 1000)]
    for kw in ({"chunk_bytes": 100}, {"lanes": 0}, {"lanes": 65}, {"tile": (3, 0)},
               {"tile": (4, 96)}, {"codebook": "tensor", "tile_order": 2}):
        with pytest.raises(wc.WcError):
            wc.encode_device_bounds(e, **kw)
    with pytest.raises(wc.WcError):
        wc.encode_device_bounds([("bf16", 1001)])
    with pytest.raises(wc.WcError):
        wc.encode_device_bounds([("u8", 1000, (3, 7))])


def test_device_encoder_rejects_before_any_launch():
    """wc_encode_device / wc_analyze_device validate every argument on the host
    before any HIP call; the fake device addresses below are never touched."""
    lib = wc.lib()
    fake = 1 << 40                      # 16-byte aligned, never dereferenced
    n = 4096
    t = (wc._Tensor * 1)(wc._Tensor(C.c_void_p(fake), n, wc.DTYPES["u8"], 0, 0, 0))
    prm = wc._Params(65536, 64, 12, 0, 0, 0, 0, 0)
    cap, wsb = wc.encode_device_bounds([("u8", n)])

    def enc(tensors=t, blob=fake, capacity=cap, ws=fake, ws_bytes=wsb, size=fake, p=prm):
        return lib.wc_encode_device(tensors, 1, C.byref(p), C.c_void_p(blob), capacity,
                                    C.c_void_p(ws), ws_bytes, None, C.c_void_p(size))

    assert enc(capacity=cap - 1) == -1          # blob one byte short
    assert enc(ws_bytes=wsb - 1) == -1          # workspace too small
    assert enc(blob=fake + 8) == -1             # misaligned blob
    assert enc(ws=fake + 4) == -1               # misaligned workspace
    assert enc(size=0) == -1                    # no size word
    assert enc(blob=0) == -1
    bad = (wc._Tensor * 1)(wc._Tensor(C.c_void_p(fake + 1), n, wc.DTYPES["u8"], 0, 0, 0))
    assert enc(tensors=bad) == -1               # misaligned source
    odd = (wc._Tensor * 1)(wc._Tensor(C.c_void_p(fake), n - 1, wc.DTYPES["bf16"], 0, 0, 0))
    assert enc(tensors=odd) == -1               # odd byte count of a 16-bit format
    assert enc(p=wc._Params(65536, 64, 11, 0, 0, 0, 0, 0)) == -1   # prob_bits must be 12
    st = wc._Stats()
    assert lib.wc_analyze_device(t, C.c_void_p(fake), wc.ANALYZE_WORKSPACE_BYTES - 1, None,
                                 C.byref(st)) == -1
    assert lib.wc_analyze_device(bad, C.c_void_p(fake), wc.ANALYZE_WORKSPACE_BYTES, None,
                                 C.byref(st)) == -1
    assert lib.wc_analyze_device(odd, C.c_void_p(fake), wc.ANALYZE_WORKSPACE_BYTES, None,
                                 C.byref(st)) == -1
