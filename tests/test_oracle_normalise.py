"""Pins for normalising counts to a 2^12 total (b = 12 probability bits, Sec. VI-F).

The rounding rule is a reading (largest remainder); it is pinned by hand-worked
cases, exact dyadic cases, invariants, and by its coding cost against the
optimal integer allocation found independently (greedy marginal gain, which is
optimal for this separable concave problem).
"""
import heapq
import math

import numpy as np
import pytest

import oracle
from paper_2606_15789_amd import synth

M = 4096


def test_dyadic_counts_are_exact():
    assert list(oracle.normalise(np.array([1, 1, 2], np.uint64))) == [1024, 1024, 2048]
    assert list(oracle.normalise(np.array([3, 0, 1], np.uint64))) == [3072, 0, 1024]
    assert list(oracle.normalise(np.array([0, 9, 0], np.uint64))) == [0, 4096, 0]


def test_hand_worked_tie_break():
    # 4096 / 3 = 1365 rem 1 for every symbol: one unit left, lowest symbol wins the tie
    assert list(oracle.normalise(np.array([1, 1, 1], np.uint64))) == [1366, 1365, 1365]
    # remainders 4096*c mod 7 for c = 1,2,4: 1, 2, 4 -> floor 585,1170,2340 (sum 4095)
    assert list(oracle.normalise(np.array([1, 2, 4], np.uint64))) == [585, 1170, 2341]


def test_forced_minimum_and_excess_removal():
    # a rare symbol rounds to 0 and is forced to 1
    assert list(oracle.normalise(np.array([1, 10 ** 6], np.uint64))) == [1, 4095]
    # 255 forced symbols push the sum to 4350; the excess comes off the largest
    h = np.ones(256, np.uint64)
    h[0] = 10 ** 9
    f = oracle.normalise(h)
    assert f[0] == 4095 - 254 and np.all(f[1:] == 1) and f.sum() == M


def test_invariants_on_random_histograms():
    rng = np.random.default_rng(11)
    for _ in range(300):
        a = int(rng.choice([2, 3, 16, 256]))
        h = rng.integers(0, 10 ** rng.integers(1, 10), size=a).astype(np.uint64)
        h[rng.random(a) < 0.4] = 0
        if h.sum() == 0:
            h[rng.integers(a)] = 1
        f = oracle.normalise(h, a)
        assert int(f.sum()) == M
        assert np.all((f > 0) == (h > 0))
        n = int(h.sum())
        # without forcing, every f is floor or ceil of the exact share
        if np.all(f[h > 0] > 1):
            exact = h.astype(np.float64) * M / n
            assert np.all(np.abs(f - exact) < 1.0 + 1e-9)


def _cost(h, f):
    return sum(int(c) * math.log2(M / int(q)) for c, q in zip(h, f) if c)


def _optimal(h):
    """Minimise sum c log2(M/f) s.t. sum f = M, f >= 1 where c > 0 (greedy is exact)."""
    f = [1 if c else 0 for c in h]
    heap = [(-float(int(c)), s) for s, c in enumerate(h) if c]   # gain of f: 1 -> 2 is c bits
    heapq.heapify(heap)
    for _ in range(M - sum(f)):
        _, s = heapq.heappop(heap)
        f[s] += 1
        heapq.heappush(heap, (-int(h[s]) * math.log2((f[s] + 1) / f[s]), s))
    return f


@pytest.mark.parametrize("which", ["bf16-exponent", "int8", "int4", "fp16-scales"])
def test_cost_close_to_optimal_allocation(which):
    if which == "bf16-exponent":
        s, _ = oracle.symbols("bf16", synth.config(2, div=8)[4].data)
    elif which == "int8":
        s, _ = oracle.symbols("u8", synth.config(4, div=8)[0].data)
    elif which == "int4":
        s, _ = oracle.symbols("u4", synth.config(3, div=8)[0].data)
    else:
        s, _ = oracle.symbols("fp16", synth.config(3, div=4)[1].data)
    a = 16 if which == "int4" else 256
    h = np.bincount(s, minlength=a).astype(np.uint64)
    n = int(h.sum())
    f = oracle.normalise(h, a)
    c_or, c_opt = _cost(h, f), _cost(h, _optimal(h))
    H = -sum(int(c) / n * math.log2(int(c) / n) for c in h if c)
    assert c_opt >= n * H - 1e-6          # Gibbs: no table beats the entropy
    assert c_or >= c_opt - 1e-6           # the greedy optimum is a lower bound
    assert (c_or - c_opt) / n < 1e-3      # within 0.001 bit/symbol of optimal
