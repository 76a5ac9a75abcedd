"""Pins for the oracle's interleaved rANS coder (Alg. 2 decode; Sec. V-B encode).

* Worked examples derived by hand from the rANS definitions (derivations in
  the comments), covering emission, the word order and the lane interleave.
* Brute force over every message up to length 6 on 2-3 symbol alphabets and
  several lane/group shapes: exact round trip, both end-of-chunk invariants,
  and agreement with a compact big-integer transcription of Duda's rANS kept
  in this file.
* The information-theoretic pin: the coded length equals the ideal length
  sum log2(2^12/f) of the message up to a per-symbol slack that the state
  interval [2^16, 2^32) bounds (see `test_code_length_bound`).
"""
import itertools
import math

import numpy as np
import pytest

import oracle

M = 4096


def test_worked_single_lane_no_emission():
    # f = {2048, 1024, 1024}, cum = {0, 2048, 3072}; encode [0,1,0,2] back to front from 65536:
    #  s=2: 65536//1024*4096 + 0 + 3072 = 265216
    #  s=0: 265216//2048*4096 + 1024     = 529408
    #  s=1: 529408//1024*4096 + 0 + 2048 = 2119680
    #  s=0: 2119680//2048*4096 + 0       = 4239360 = 0x40B000
    f = [2048, 1024, 1024]
    st, w = oracle.encode_stream([0, 1, 0, 2], f, 1, 1)
    assert list(st) == [0x40B000] and len(w) == 0
    assert list(oracle.decode_stream(st, w, 4, f, 1, 1)) == [0, 1, 0, 2]


def test_worked_emissions():
    # f = {4095, 1}.  [1,1,1]: 65536 -> 0x10000FFF; emit 0x0FFF -> 0x1000 -> 0x1000FFF;
    # emit 0x0FFF -> 0x100 -> 0x100FFF.  Stack [0FFF, 0FFF] read top first.
    f = [4095, 1]
    st, w = oracle.encode_stream([1, 1, 1], f, 1, 1)
    assert list(st) == [1052671] and list(w) == [0x0FFF, 0x0FFF]
    # [1,0,1,1]: ... 0x1000FFF; s=0: 16781311 = 4098*4095 + 1 -> 4098*4096 + 1 = 0x1002001;
    # s=1: emit 0x2001, 0x100 -> 0x100FFF.  Stack [0FFF, 2001] -> stream [2001, 0FFF].
    st, w = oracle.encode_stream([1, 0, 1, 1], f, 1, 1)
    assert list(st) == [1052671] and list(w) == [0x2001, 0x0FFF]
    assert list(oracle.decode_stream(st, w, 4, f, 1, 1)) == [1, 0, 1, 1]


def test_worked_two_lanes_group_two():
    # 2 lanes, W = 2: symbol i -> lane (i mod 4) div 2, step (i div 4)*2 + i mod 2.
    # lane 0 gets [1,0,0,1], lane 1 gets [1,1,1,1].  Back to front per step, lane 1 first:
    #  lane 1: 0x10000FFF; emit 0FFF ->0x1000FFF; emit 0FFF ->0x100FFF; emit 0FFF -> 0x10FFF
    #  lane 0: 0x10000FFF; s=0 -> 268505104; s=0 -> 268570673 = 4098*65536 + 0x1031;
    #          emit 0x1031 -> 4098 -> 0x1002FFF
    # pushes: t=2 lane1, t=1 lane1, t=0 lane1, t=0 lane0 -> stream [1031, 0FFF, 0FFF, 0FFF]
    f = [4095, 1]
    msg = [1, 0, 1, 1, 0, 1, 1, 1]
    st, w = oracle.encode_stream(msg, f, 2, 2)
    assert list(st) == [0x1002FFF, 0x10FFF]
    assert list(w) == [0x1031, 0x0FFF, 0x0FFF, 0x0FFF]
    assert list(oracle.decode_stream(st, w, 8, f, 2, 2)) == msg


def test_single_symbol_table_emits_nothing():
    st, w = oracle.encode_stream([0] * 1000, [4096], 64, 4)
    assert np.all(st == 65536) and len(w) == 0


# ---------------------------------------------------------------------------
# Big-integer transcription of Duda's streaming rANS (state in [L, L*2^16),
# 16-bit words, probabilities f/M), with the lane/step assignment of the
# format.  Written independently of wc_oracle.c.

def duda(msg, f, lanes, group):
    cum = [sum(f[:s]) for s in range(len(f))]
    n = len(msg)
    owner = {}
    for i in range(n):
        row, r = divmod(i, lanes * group)
        owner[i] = (r // group, row * group + r % group)
    A = min(lanes, -(-n // group))
    x = [1 << 16] * A
    pushes = []
    for i in sorted(range(n), key=lambda i: (owner[i][1], owner[i][0]), reverse=True):
        lane, s = owner[i][0], msg[i]
        if x[lane] >= f[s] << 20:
            pushes.append(x[lane] % 65536)
            x[lane] //= 65536
        x[lane] = M * (x[lane] // f[s]) + cum[s] + x[lane] % f[s]
    return x, pushes[::-1]


TABLES = [[2048, 2048], [4095, 1], [1, 4095], [1, 1, 4094], [2048, 1024, 1024], [3000, 1000, 96]]
SHAPES = [(1, 1), (2, 2), (3, 1), (2, 4), (64, 2), (64, 8), (32, 4)]


@pytest.mark.parametrize("f", TABLES)
def test_brute_force_small_messages(f):
    a = len(f)
    for length in range(1, 7):
        for msg in itertools.product(range(a), repeat=length):
            for lanes, group in SHAPES:
                st, w = oracle.encode_stream(list(msg), f, lanes, group)
                x, words = duda(list(msg), f, lanes, group)
                assert list(st) == x and list(w) == words, (msg, lanes, group)
                back = oracle.decode_stream(st, w, length, f, lanes, group)
                assert tuple(back) == msg


def _check_length(msg, f, lanes, group):
    st, w = oracle.encode_stream(msg, f, lanes, group)
    used = 16 * len(w) + sum(math.log2(int(v)) for v in st) - 16 * len(st)
    ideal = sum(math.log2(M / f[s]) for s in msg)
    return used, ideal


def test_code_length_bound():
    # Each encode maps x in [16 f, 2^20 f) to C with |C - x M/f| < M <= (x M/f)/16, i.e.
    # at most log2(16/15) bits away from the ideal; each emission of the word w from
    # x = h*2^16 + w (h >= 16) loses at most log2(17/16) bits.  So
    # |bits used - ideal| <= n * (log2(16/15) + log2(17/16)) for any message.
    slack = math.log2(16 / 15) + math.log2(17 / 16)
    rng = np.random.default_rng(3)
    for _ in range(40):
        a = int(rng.choice([2, 5, 16, 256]))
        h = rng.integers(1, 1000, size=a).astype(np.uint64)
        f = [int(v) for v in oracle.normalise(h, a)]
        n = int(rng.integers(1, 3000))
        p = np.array(f) / M
        msg = [int(s) for s in rng.choice(a, size=n, p=p)]
        for lanes, group in [(1, 1), (64, 2), (32, 4)]:
            used, ideal = _check_length(msg, f, lanes, group)
            assert abs(used - ideal) <= n * slack + 1e-6
    # and on long typical messages the excess is tiny
    f = [int(v) for v in oracle.normalise(np.array([900, 50, 40, 10] * 4, np.uint64), 16)]
    msg = [int(s) for s in rng.choice(16, size=200_000, p=np.array(f) / M)]
    used, ideal = _check_length(msg, f, 1, 1)
    assert abs(used - ideal) / len(msg) < 0.005


def test_corrupted_word_or_state_is_detected():
    rng = np.random.default_rng(9)
    f = [int(v) for v in oracle.normalise(np.array([500, 300, 150, 50], np.uint64), 4)]
    msg = rng.choice(4, size=5000, p=np.array(f) / M).astype(np.uint8)
    st, w = oracle.encode_stream(msg, f, 64, 2)
    assert np.array_equal(oracle.decode_stream(st, w, msg.size, f, 64, 2), msg)
    bad = w.copy()
    bad[len(bad) // 2] ^= 0x0100
    with pytest.raises(oracle.OracleError) as e:
        oracle.decode_stream(st, bad, msg.size, f, 64, 2)
    assert e.value.rc == -3
    st2 = st.copy()
    st2[5] += 1
    with pytest.raises(oracle.OracleError):
        oracle.decode_stream(st2, w, msg.size, f, 64, 2)
    with pytest.raises(oracle.OracleError):   # truncated stream
        oracle.decode_stream(st, w[:-1], msg.size, f, 64, 2)
