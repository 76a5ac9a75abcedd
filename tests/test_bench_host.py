"""CPU checks of bench.py's host logic: the one-GPU guard, and the rules by
which it names the kernel a launch runs on (the library takes the same
decision from the runtime's occupancy figures; a 256-CU MI355X holds 24 waves
of the 8-wave kernels and 32 of the 16-wave ones per compute unit)."""
import importlib.util
import os
import subprocess
import sys
import types

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def bench():
    spec = importlib.util.spec_from_file_location("bench_under_test", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


@pytest.fixture
def cus_256(monkeypatch):
    torch = pytest.importorskip("torch")
    monkeypatch.setattr(torch.cuda, "get_device_properties",
                        lambda dev: types.SimpleNamespace(multi_processor_count=256))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU only" in r.stderr
    assert r.stdout == ""


@pytest.mark.parametrize("chunks,wide", [(6144, False), (6145, True), (8192, True), (8193, False)])
def test_decode_kernel_window(bench, cus_256, chunks, wide):
    want = "wc_decode_wide_kernel" if wide else "wc_decode_kernel"
    assert bench.decode_kernel_for(["bf16"] * 7, chunks, 64, False) == want
    assert bench.decode_kernel_for(["fp16", "bf16"], chunks, 64, False) == want


def test_decode_kernel_window_needs_untiled_16_bit_64_lane_launches(bench, cus_256):
    assert bench.decode_kernel_for(["bf16"], 7000, 64, True) == "wc_decode_kernel"
    assert bench.decode_kernel_for(["bf16"], 7000, 32, False) == "wc_decode_kernel"
    assert bench.decode_kernel_for(["bf16", "u8"], 7000, 64, False) == "wc_decode_kernel"


@pytest.mark.parametrize("weights,rows", [("bf16", 16), ("int8", 16), ("e4m3", 16), ("e5m2", 16),
                                          ("mxfp4-bytes", 8), ("int4-bytes", 8)])
def test_gemv_kernel_window(bench, cus_256, weights, rows):
    inside = bench.gemv_kernel_for(weights, 6656, rows)
    assert "wide" in inside
    assert "wide" in bench.gemv_kernel_for(weights, 8192, 1)
    for tiles, m in [(6144, 1), (8193, 1), (6656, rows + 1)]:
        name = bench.gemv_kernel_for(weights, tiles, m)
        assert "wide" not in name and name.startswith("wc_gemv_"), (tiles, m, name)


def test_nibble_coded_4_bit_codes_keep_the_8_wave_kernels(bench, cus_256):
    assert bench.gemv_kernel_for("mxfp4", 6656, 1) == "wc_gemv_mx_kernel"
    assert bench.gemv_kernel_for("int4", 6656, 1) == "wc_gemv_w4n_kernel"


def test_counted_traffic_only_for_the_kernel_and_layout_it_was_taken_on(bench, monkeypatch):
    for workload, c in bench.COUNTED_TRAFFIC.items():
        prints = {c["kernel"]: c["kernel_fingerprint"]}
        monkeypatch.setattr(bench, "kernel_fingerprint", lambda name: prints.get(name))
        want = c["fetch_bytes"] + c["write_bytes"]
        assert bench.counted_traffic(workload, 65536, 64, False, c["kernel"]) == want
        assert bench.counted_traffic(workload, 32768, 64, False, c["kernel"]) is None
        assert bench.counted_traffic(workload, 65536, 32, False, c["kernel"]) is None
        assert bench.counted_traffic(workload, 65536, 64, True, c["kernel"]) is None
        other = "wc_decode_kernel" if c["kernel"] != "wc_decode_kernel" else "wc_decode_wide_kernel"
        assert bench.counted_traffic(workload, 65536, 64, False, other) is None
        prints[c["kernel"]] = "0000000000000000"          # the kernel's code changed
        assert bench.counted_traffic(workload, 65536, 64, False, c["kernel"]) is None
    assert bench.counted_traffic("bf16-matrix-4096", 65536, 64, False, "wc_decode_kernel") is None
