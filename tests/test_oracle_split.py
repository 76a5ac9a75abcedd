"""Pins for the oracle's field split (the storage format fixes the symbols, Sec. II-B).

The split of a 16-bit float word into a coded exponent byte and a raw
sign|mantissa byte is pinned against IEEE semantics through library routines
(torch's float->bfloat16 rounding, math.frexp), not against a retyped copy of
the bit formula.
"""
import math

import numpy as np
import pytest
import torch

import oracle


def bf16_bits(x: float) -> int:
    return int(torch.tensor([x], dtype=torch.float32).to(torch.bfloat16).view(torch.int16)[0]) & 0xFFFF


@pytest.mark.parametrize("x,word,coded,raw", [
    (1.0, 0x3F80, 0x7F, 0x00),
    (-0.02, 0xBCA4, 0x79, 0xA4),
    (0.02, 0x3CA4, 0x79, 0x24),
    (-1.5, 0xBFC0, 0x7F, 0xC0),
])
def test_split_worked_values(x, word, coded, raw):
    # bf16 rounding by torch (RNE), then the split.
    assert bf16_bits(x) == word
    assert oracle.coded16(word) == coded
    assert oracle.raw16(word) == raw
    assert oracle.merge16(coded, raw) == word


def _bf16_values(words: np.ndarray) -> np.ndarray:
    with np.errstate(invalid="ignore"):
        return (words.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def test_split_is_ieee_exponent_and_sign_mantissa_bf16():
    """coded byte = biased exponent, raw = sign bit + 7 mantissa bits, for all 2^16 patterns."""
    words = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    coded, raw = oracle.symbols("bf16", words)
    vals = _bf16_values(words)
    for w in range(65536):
        v = vals[w]
        c, r = int(coded[w]), int(raw[w])
        assert (r >> 7) == int(math.copysign(1.0, v) < 0), hex(w)
        if math.isnan(v) or math.isinf(v):
            assert c == 255
            continue
        if v == 0.0 or abs(v) < 2.0 ** -126:   # zero / subnormal
            assert c == 0 and (c & 1) == 0
            continue
        m, e = math.frexp(abs(v))            # |v| = m * 2^e, 0.5 <= m < 1
        assert c == e - 1 + 127, hex(w)
        frac = abs(v) / 2.0 ** (e - 1) - 1.0  # in [0, 1), exact
        assert (r & 0x7F) == int(frac * 128), hex(w)


def test_split_fp16_uses_same_bit_positions():
    """fp16: coded = 5-bit exponent followed by the top 3 mantissa bits; raw = sign + low 7."""
    words = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    coded, raw = oracle.symbols("fp16", words)
    vals = words.view(np.float16).astype(np.float64)
    for w in range(0, 65536, 7):
        v = vals[w]
        c, r = int(coded[w]), int(raw[w])
        assert (r >> 7) == int(math.copysign(1.0, v) < 0)
        if math.isnan(v) or math.isinf(v) or v == 0.0 or abs(v) < 2.0 ** -14:
            continue
        m, e = math.frexp(abs(v))
        mant10 = int((abs(v) / 2.0 ** (e - 1) - 1.0) * 1024)
        assert (c >> 3) == e - 1 + 15
        assert (c & 7) == mant10 >> 7
        assert (r & 0x7F) == mant10 & 0x7F


def test_merge_inverts_split_on_every_pattern():
    words = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    coded, raw = oracle.symbols("bf16", words)
    back = np.array([oracle.merge16(int(c), int(r)) for c, r in zip(coded, raw)], np.uint16)
    assert np.array_equal(back, words)


def test_int8_and_int4_symbols():
    b = np.arange(256, dtype=np.uint8)
    s8, r8 = oracle.symbols("u8", b)
    assert r8 is None and np.array_equal(s8, b)
    s4, r4 = oracle.symbols("u4", b)
    assert r4 is None
    # two's complement int4 pair packed low nibble first
    assert np.array_equal(s4[0::2], b & 0x0F)
    assert np.array_equal(s4[1::2], b >> 4)
    q = np.array([-8, 7, -1, 0], dtype=np.int8)
    packed = ((q[0::2].view(np.uint8) & 0xF) | ((q[1::2].view(np.uint8) & 0xF) << 4)).astype(np.uint8)
    s, _ = oracle.symbols("u4", packed)
    assert list(s) == [8, 7, 15, 0]
