"""GPU parity on randomised blobs: the decode kernel against the oracle.

A seeded generator draws 120 blobs of one to five tensors: every storage
format, sizes from empty to a few thousand elements (ragged tails, chunks of
a few symbols, lanes left empty), flat, peaked or single-symbol value
distributions, chunk sizes from 256 bytes to 64 KiB, 64 or 32 lanes (the
decoder's two shapes), byte-run chunks or 2-D tiles in either order with a
per-tensor or layer codebook.  Each blob is encoded by the host library,
decoded by wc_decode through the C ABI, and must equal the original bytes and
the oracle's decode of the same blob, with no error bit set.
"""
import sys

import numpy as np
import pytest

import oracle
from paper_2606_15789_amd import wc

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

DTYPES = ["bf16", "fp16", "u8", "u4", "fp8_e4m3", "fp8_e5m2", "fp4_e2m1"]


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda:0")


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _tensor(rng, dt, n_bytes, skew):
    if dt in ("bf16", "fp16"):
        n = n_bytes // 2
        if skew == 0:
            return np.full(n, 0xBC80, np.uint16)
        w = rng.normal(0, 0.02 if skew == 1 else 3.0, n).astype(np.float32)
        return (w.view(np.uint32) >> 16).astype(np.uint16)
    if skew == 0:
        return np.full(n_bytes, 0xA7, np.uint8)
    if skew == 1:
        return np.clip(rng.normal(100, 5, n_bytes), 0, 255).astype(np.uint8)
    return rng.integers(0, 256, n_bytes).astype(np.uint8)


def _case(rng):
    tile = [(0, 0), (16, 64), (32, 128), (64, 256)][rng.integers(0, 4)]
    order = int(rng.integers(0, 2))
    codebook = ["tensor", "layer"][rng.integers(0, 2)]
    lanes = [64, 32][rng.integers(0, 2)]
    chunk = int(256 * rng.choice([1, 3, 16, 64, 256]))
    entries = []
    for _ in range(int(rng.integers(1, 6))):
        dt = DTYPES[rng.integers(0, len(DTYPES))]
        skew = int(rng.integers(0, 3))
        if tile != (0, 0) and rng.random() < 0.5:
            rows, cols = tile[0] * int(rng.integers(1, 3)), tile[1] * int(rng.integers(1, 3))
            n_sym = rows * cols
            nb = 2 * n_sym if dt in ("bf16", "fp16") else (n_sym // 2 if dt in ("u4", "fp4_e2m1")
                                                           else n_sym)
            entries.append((dt, _tensor(rng, dt, nb, skew), (rows, cols)))
        else:
            nb = int(rng.integers(0, 9000))
            nb -= nb % 2 if dt in ("bf16", "fp16") else 0
            entries.append((dt, _tensor(rng, dt, nb, skew)))
    return entries, dict(chunk_bytes=chunk, lanes=lanes, tile=tile, codebook=codebook,
                         tile_order=order)


def test_random_blobs_decode_like_the_oracle(dev):
    rng = np.random.default_rng(260615789)
    err = torch.zeros(1, dtype=torch.int32, device=dev)
    for i in range(120):
        entries, kw = _case(rng)
        say(f"random blob {i}: {[(e[0], np.asarray(e[1]).nbytes) for e in entries]} {kw}")
        blob = wc.encode(entries, threads=2, **kw)
        ref = oracle.decode(blob.tobytes())
        d = wc.to_device(blob, dev)
        err.zero_()
        outs = wc.decode_torch(blob, d, err=err)
        torch.cuda.synchronize()
        assert int(err.item()) == 0, (i, wc.describe_errors(int(err.item())))
        for t, (e, out, r) in enumerate(zip(entries, outs, ref)):
            got = out.cpu().numpy()
            orig = np.ascontiguousarray(e[1]).view(np.uint8).reshape(-1)
            assert np.array_equal(got, orig), (i, t)
            assert np.array_equal(got, r), (i, t)
