"""The C ABI from plain C: paper_2606_15789_amd/csrc/wc_example.c, built next
to the library, allocates with hipMalloc, encodes on the host, decodes on the
GPU (bit-exact) and runs the fused decode-GEMV (fp32 summation bound against
its own fp64 dot products), with no Python or PyTorch in the process."""
import os
import subprocess

import pytest

from paper_2606_15789_amd import build

pytestmark = pytest.mark.gpu


def test_plain_c_client():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    exe = build.ensure_example()
    assert os.path.exists(exe)
    r = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, (r.stdout, r.stderr)
    assert "bit-exact" in r.stdout and "matches fp64" in r.stdout, r.stdout
