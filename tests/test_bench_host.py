"""Host-side logic of bench.py and of the counter summaries it reads (no GPU)."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_2602_03839_amd import traffic  # noqa: E402


def test_counter_bound_reproduces_its_two_streams():
    # a launch that moves exactly the read stream's bytes takes fetch / read rate
    cb = bench.counter_bound((6.0e9, 0.0), 6000.0, 4000.0, 1.0)
    assert cb["bound_ms"] == pytest.approx(1.0)
    assert cb["frac"] == pytest.approx(1.0)
    # a launch with the read-modify-write stream's mix (8 B read, 4 B written
    # per element) runs at that stream's rate
    n = 1.0e9
    cb = bench.counter_bound((8.0 * n, 4.0 * n), 6000.0, 4000.0, 3.0)
    assert cb["bound_ms"] == pytest.approx(12.0 * n / 4000e9 * 1e3)
    # written bytes cost more than read ones whenever the rmw stream is slower
    assert cb["write_marginal_GBps"] < 6000.0


def test_traffic_summary_split_and_source_hash(tmp_path):
    good = tmp_path / "good.txt"
    good.write_text(f"# header: with a colon\nsource_hash: {traffic.kernel_source_hash()}\n"
                    "fetch_bytes_per_launch: 100\nwrite_bytes_per_launch: 23\n")
    assert traffic.read_summary_split(str(good)) == (100.0, 23.0)
    assert traffic.read_summary(str(good)) == 123.0
    stale = tmp_path / "stale.txt"
    stale.write_text("source_hash: 0000000000000000\nfetch_bytes_per_launch: 1\nwrite_bytes_per_launch: 1\n")
    assert traffic.read_summary_split(str(stale)) is None
    assert traffic.read_summary(str(tmp_path / "missing.txt")) is None


def test_kernel_labels():
    assert traffic.kernel_label("void pulse::(anonymous namespace)::outer_kernel(pulse::OuterParams)") == \
        "outer_kernel"
    assert traffic.kernel_label("void pulse::encode_kernel<15, 2, true>(pulse::EncodeParams)") == \
        "encode_kernel<15, 2, true>"


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode != 0
    assert "one GPU" in (r.stdout + r.stderr)
