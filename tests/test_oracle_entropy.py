"""Pins for the oracle's empirical entropy (Sec. II-B, per-tensor H and the bound).

Closed forms (uniform, single symbol) and scipy's entropy routine fix the
value; the joint 16-bit entropy is tied to the field entropies by the
subadditivity and monotonicity inequalities of Shannon entropy.
"""
import math

import numpy as np
import pytest
import scipy.stats

import oracle
from paper_2606_15789_amd import synth


@pytest.mark.parametrize("k", range(0, 9))
def test_uniform_power_of_two(k):
    h = np.zeros(256, np.uint64)
    h[: 2 ** k] = 37
    assert oracle.entropy(h) == pytest.approx(float(k), abs=1e-12)


def test_single_symbol_and_empty():
    h = np.zeros(256, np.uint64)
    h[200] = 12345
    assert oracle.entropy(h) == 0.0
    assert oracle.entropy(np.zeros(256, np.uint64)) == 0.0


@pytest.mark.parametrize("p", [0.5, 0.1, 0.01, 0.9999])
def test_binary_entropy(p):
    n = 1_000_000
    c1 = int(round(p * n))
    h = np.zeros(16, np.uint64)
    h[3], h[11] = c1, n - c1
    q = c1 / n
    closed = -(q * math.log2(q) + (1 - q) * math.log2(1 - q))
    assert oracle.entropy(h, 16) == pytest.approx(closed, rel=1e-12)


def test_matches_scipy_on_random_histograms():
    rng = np.random.default_rng(5)
    for _ in range(50):
        a = int(rng.choice([16, 256]))
        h = rng.integers(0, 10 ** rng.integers(1, 9), size=a).astype(np.uint64)
        h[rng.random(a) < 0.3] = 0
        if h.sum() == 0:
            h[0] = 1
        ref = scipy.stats.entropy(h.astype(np.float64), base=2)
        assert oracle.entropy(h, a) == pytest.approx(ref, rel=1e-10, abs=1e-12)


def test_analyze_bf16_fields_and_joint():
    w = synth.config(1, div=8)[0].data
    st = oracle.analyze("bf16", w)
    coded, raw = oracle.symbols("bf16", w)
    n = w.size
    ref_c = scipy.stats.entropy(np.bincount(coded, minlength=256), base=2)
    ref_r = scipy.stats.entropy(np.bincount(raw, minlength=256), base=2)
    ref_j = scipy.stats.entropy(np.unique(w, return_counts=True)[1], base=2)
    assert st["count"] == [n, n]
    assert st["H"][0] == pytest.approx(ref_c, rel=1e-10)
    assert st["H"][1] == pytest.approx(ref_r, rel=1e-10)
    assert st["H_joint16"] == pytest.approx(ref_j, rel=1e-10)
    # H(X,Y) <= H(X) + H(Y) and H(X,Y) >= max(H(X), H(Y))
    assert st["H_joint16"] <= st["H"][0] + st["H"][1] + 1e-9
    assert st["H_joint16"] >= max(st["H"]) - 1e-9
    assert st["bound_bytes"] == pytest.approx(n * (st["H"][0] + st["H"][1]) / 8, rel=1e-12)
    assert st["bound_bytes_raw8"] == pytest.approx(n * st["H"][0] / 8 + n, rel=1e-12)
    # N(0, 0.02) in bf16: the exponent carries ~2.5 bits, sign+mantissa ~8
    assert 2.3 < st["H"][0] < 2.8 and 7.9 < st["H"][1] <= 8.0


def test_analyze_int4_and_int8():
    ts = synth.config(3, div=16)
    q = [t for t in ts if t.dtype == "u4"][0]
    st = oracle.analyze("u4", q.data)
    s, _ = oracle.symbols("u4", q.data)
    assert st["n_fields"] == 1 and st["alphabet"] == [16]
    assert st["H"][0] == pytest.approx(scipy.stats.entropy(np.bincount(s, minlength=16), base=2))
    assert math.isnan(st["H_joint16"])
    assert st["H"][0] <= 4.0
