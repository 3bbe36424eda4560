"""Host-side logic of bench.py (no GPU): the one-GPU contract, the
algorithmic byte count behind the roofline figure, and the rule that stored
counter traffic is only reported for the kernel sources it was taken on."""

import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_more_than_one_gpu_is_refused():
    res = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                         text=True, timeout=120)
    assert res.returncode == 2
    assert "one GPU" in res.stderr and res.stdout == ""


def test_algorithmic_bytes_per_row():
    # one read of a V = 151,936 bf16 row, the sampled id and temperature in, ten 4-byte outputs
    assert bench.algorithmic_bytes_per_row(151936, 2) == 151936 * 2 + 8 + 40
    assert bench.algorithmic_bytes_per_row(262144, 4) == (1 << 20) + 48


def test_kernel_sources_exist_and_hash_is_stable():
    for kernel, files in bench.KERNEL_SOURCES.items():
        for fn in files:
            assert os.path.exists(os.path.join(ROOT, fn)), fn
        h = bench.kernel_source_hash(kernel)
        assert len(h) == 16 and h == bench.kernel_source_hash(kernel)


@pytest.mark.parametrize("path,key", [("features", "w"), ("sample", "w:sample")])
def test_stored_traffic_needs_the_same_kernel_sources(tmp_path, path, key):
    tj = tmp_path / "traffic.json"
    good = {"kernel": "row_features_kernel", "bytes_per_launch": 123.0,
            "kernel_source_hash": bench.kernel_source_hash("row_features_kernel")}
    tj.write_text(json.dumps({key: good}))
    assert bench.stored_traffic(str(tj), "w", path) == 123.0
    assert bench.stored_traffic(str(tj), "other", path) is None
    tj.write_text(json.dumps({key: dict(good, kernel_source_hash="0" * 16)}))
    assert bench.stored_traffic(str(tj), "w", path) is None          # taken on other sources
    tj.write_text(json.dumps({key: dict(good, kernel="no_such_kernel")}))
    assert bench.stored_traffic(str(tj), "w", path) is None
    tj.write_text("not json")
    assert bench.stored_traffic(str(tj), "w", path) is None
    assert bench.stored_traffic(str(tmp_path / "missing.json"), "w", path) is None


def test_committed_traffic_records_name_known_kernels():
    d = json.load(open(os.path.join(ROOT, "profiles", "traffic.json")))
    for key, t in d.items():
        assert t["kernel"] in bench.KERNEL_SOURCES, key
        assert t["bytes_per_launch"] > 0 and t["fetch_scale"] > 0 and t["write_scale"] > 0, key
