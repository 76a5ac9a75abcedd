"""GPU: wc_stream, the streaming kernel that the decode's throughput is set
against.  It must move exactly the bytes it says it moves: write unit j of dst
is read unit (j * q) >> 32 of src, q = floor(n_src * 2^32 / n_dst), every unit
of src up to the last index it reports is read, and nothing past dst is
written."""
import sys

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


@pytest.mark.parametrize("n_src,n_dst,blocks", [(1, 1, 0), (1000, 1517, 0), (1517, 1517, 3),
                                                (4099, 65537, 7), (3, 100003, 0),
                                                (4_000_000, 6_000_001, 0)])
def test_stream_moves_the_stated_units(dev, n_src, n_dst, blocks):
    say(f"wc_stream n_src={n_src} n_dst={n_dst} blocks={blocks}")
    g = torch.Generator(device=dev)
    g.manual_seed(n_src * 7 + n_dst)
    src = torch.randint(-2**31, 2**31 - 1, (n_src, 4), generator=g, dtype=torch.int32,
                        device=dev)
    guard = 64
    dst = torch.full((n_dst + guard, 4), -1, dtype=torch.int32, device=dev)
    read = wc.stream_bytes(src.data_ptr(), 16 * n_src, dst.data_ptr(), 16 * n_dst, blocks,
                           torch.cuda.current_stream(dev).cuda_stream)
    torch.cuda.synchronize()
    q = (n_src << 32) // n_dst
    j = torch.arange(n_dst, dtype=torch.int64, device=dev)
    r = (j * q) >> 32                                    # < 2^63 for these sizes
    assert int(r.max()) < n_src
    assert read == 16 * (int(r.max()) + 1)
    assert read >= 16 * (n_src - 2)                    # the whole source, but for rounding
    assert torch.equal(dst[:n_dst], src[r])
    assert bool((dst[n_dst:] == -1).all())              # nothing past dst


def test_stream_read_only(dev):
    n_src = 1_000_003
    src = torch.arange(4 * n_src, dtype=torch.int32, device=dev).view(n_src, 4)
    sink = torch.full((4,), 7, dtype=torch.int32, device=dev)
    read = wc.stream_bytes(src.data_ptr(), 16 * n_src, sink.data_ptr(), 0)
    torch.cuda.synchronize()
    assert read == 16 * n_src
    # each thread's XOR of these small integers stays below 2^23: never the pattern
    assert sink.tolist() == [7, 7, 7, 7]
