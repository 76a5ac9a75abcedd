"""CPU: randomised agreement of the library's host encoder with the oracle.

Hypothesis draws blobs of one to four tensors with every storage format, sizes
from empty to a few thousand elements, skewed or flat value distributions
(single-symbol tensors included), chunk sizes from 256 bytes, 1 to 64 lanes,
and, for shaped tensors, 2-D tiles in either tile order with a per-tensor or
layer codebook.  For every draw the library's blob must equal the oracle's
byte for byte, the oracle must decode it back to the input, and wc_open must
accept it with the same per-tensor sizes.  No GPU call is made.
"""
import numpy as np
import pytest
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

import oracle
from paper_2606_15789_amd import wc

DTYPES = ["bf16", "fp16", "u8", "u4", "fp8_e4m3", "fp8_e5m2", "fp4_e2m1"]
ELEM_BYTES = {"bf16": 2, "fp16": 2}


def _values(rng, dtype, n_bytes, skew):
    """Storage bytes of one tensor: flat, or geometric-like (many rare symbols)."""
    if dtype in ("bf16", "fp16"):
        n = n_bytes // 2
        if skew == "one":
            return np.full(n, 0x3F80, np.uint16)
        w = rng.normal(0, 0.02 if skew == "normal" else 1.0, n).astype(np.float32)
        return (w.view(np.uint32) >> 16).astype(np.uint16)
    if skew == "one":
        return np.full(n_bytes, 0x5A, np.uint8)
    if skew == "normal":
        return np.clip(rng.normal(128, 6, n_bytes), 0, 255).astype(np.uint8)
    return rng.integers(0, 256, n_bytes).astype(np.uint8)


@st.composite
def blobs(draw):
    seed = draw(st.integers(0, 2**31 - 1))
    rng = np.random.default_rng(seed)
    n_t = draw(st.integers(1, 4))
    tile = draw(st.sampled_from([(0, 0), (16, 64), (32, 128), (8, 32)]))
    order = draw(st.integers(0, 1))
    codebook = draw(st.sampled_from(["tensor", "layer"]))
    entries = []
    for _ in range(n_t):
        dt = draw(st.sampled_from(DTYPES))
        skew = draw(st.sampled_from(["one", "normal", "flat"]))
        shaped = draw(st.booleans()) and tile != (0, 0)
        if shaped:
            # rows x cols in symbol elements, multiples of the tile
            rows = tile[0] * draw(st.integers(1, 3))
            cols = tile[1] * draw(st.integers(1, 3))
            n_sym = rows * cols
            n_bytes = n_sym * 2 if dt in ELEM_BYTES else (n_sym // 2 if dt in ("u4", "fp4_e2m1")
                                                          else n_sym)
            entries.append((dt, _values(rng, dt, n_bytes, skew), (rows, cols)))
        else:
            n_bytes = draw(st.integers(0, 6000))
            if dt in ELEM_BYTES:
                n_bytes -= n_bytes % 2
            entries.append((dt, _values(rng, dt, n_bytes, skew)))
    chunk = 256 * draw(st.integers(1, 16))
    lanes = draw(st.sampled_from([1, 2, 7, 16, 32, 63, 64]))
    return entries, chunk, lanes, tile, order, codebook


@settings(max_examples=120, deadline=None, suppress_health_check=[HealthCheck.too_slow])
@given(blobs())
def test_random_blobs_identical_to_oracle(case):
    entries, chunk, lanes, tile, order, codebook = case
    kw = dict(chunk_bytes=chunk, lanes=lanes, tile=tile, codebook=codebook, tile_order=order)
    ref = oracle.encode(entries, **kw)
    got = wc.encode(entries, threads=3, **kw)
    assert got.tobytes() == ref
    outs = oracle.decode(ref)
    for e, o in zip(entries, outs):
        assert np.array_equal(o, np.ascontiguousarray(e[1]).view(np.uint8).reshape(-1))
    opened = wc.open_blob(ref)
    assert opened.out_bytes == [int(np.asarray(e[1]).nbytes) for e in entries]
    assert opened.size == got.size
