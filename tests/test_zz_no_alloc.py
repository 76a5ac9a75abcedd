"""GPU: wc_analyze_device_static, the analysis entry point that allocates
nothing (its histogram bins are the library's own device array), against
wc_analyze_device with a caller workspace and against the host wc_analyze.

Calls follow one another on the same array: a large tensor, then a smaller
one, then other formats, so that anything a call left in the bins would show
up in the next call's counts."""
import math
import sys
import threading

import numpy as np
import pytest

from paper_2606_15789_amd import wc

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


def _same(a: dict, b: dict):
    """Every field equal, the histograms bin for bin, the entropies to the bit
    (NaN where both are NaN)."""
    assert a.keys() == b.keys()
    for k in a:
        x, y = a[k], b[k]
        if k == "hist":
            assert len(x) == len(y)
            for u, v in zip(x, y):
                assert np.array_equal(u, v), k
        elif isinstance(x, list):
            assert [float(u).hex() if isinstance(u, float) else u for u in x] == \
                [float(v).hex() if isinstance(v, float) else v for v in y], k
        elif isinstance(x, float):
            assert (math.isnan(x) and math.isnan(y)) or x.hex() == y.hex(), k
        else:
            assert x == y, k


def _cases():
    rng = np.random.default_rng(355)
    bf = lambda n: (rng.normal(0, 0.02, n).astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)  # noqa: E731
    return [
        ("bf16", bf(3_000_001)),                                         # large first
        ("bf16", bf(1001)),                                              # then smaller
        ("u8", rng.integers(0, 256, 77_777).astype(np.uint8)),
        ("fp16", rng.normal(0, 1, 4097).astype(np.float16).view(np.uint16)),
        ("u4", rng.integers(0, 256, 5000).astype(np.uint8)),
        ("fp8_e4m3", rng.integers(0, 256, 31).astype(np.uint8)),
        ("bf16", np.zeros(0, np.uint16)),                                # empty
        ("bf16", bf(65_536)),
    ]


def test_static_analysis_matches_workspace_analysis(dev):
    for i, (dt, h) in enumerate(_cases()):
        say(f"analyze_device_static case {i}: {dt} {h.size} elements")
        x = torch.from_numpy(h.view(np.uint8).copy()).to(dev)
        got = wc.analyze_device_static(dt, x)
        ref = wc.analyze_device(dt, x)
        _same(got, ref)
        _same(got, wc.analyze(dt, h))


def test_static_analysis_from_several_host_threads(dev):
    """Host threads calling at once take turns on the one array."""
    cases = _cases()[:6]
    xs = [torch.from_numpy(h.view(np.uint8).copy()).to(dev) for _, h in cases]
    refs = [wc.analyze(dt, h) for dt, h in cases]
    results, errors = {}, []

    def work(k):
        try:
            torch.cuda.set_device(dev)
            for j in range(3):
                i = (k + j) % len(cases)
                results[(k, j)] = (i, wc.analyze_device_static(cases[i][0], xs[i]))
        except Exception as e:  # noqa: BLE001
            errors.append(e)

    threads = [threading.Thread(target=work, args=(k,)) for k in range(4)]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    assert not errors, errors
    assert len(results) == 12
    for i, st in results.values():
        _same(st, refs[i])
