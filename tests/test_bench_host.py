"""Host-side pieces of bench.py: the algorithmic byte count behind roofline.achieved,
the profile lookup behind roofline.traffic, the head-pair report and the argument
contract (no GPU needed)."""
import os
import subprocess
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def test_algorithmic_bytes_closed_form():
    # two rows, 1000 and 17 tokens, Hq = 32, Hkv = 8, d = 128, 12 tasks
    lens = [1000, 17]
    total, kv = bench.algorithmic_bytes(lens, 12)
    assert kv == 4096 * 1017                              # K and V, 8 heads x 128 dims x 2 B each
    qo = 2 * 2 * 32 * 128 * 2                             # Q read and out written, fp16
    meta = 4 * (63 + 2) + 4 * 2 + 4 * 3 + 20 * 12         # page ids, lengths, offsets, task records
    partial = 2 * 2080 * 12                               # each partial state written and read once
    assert total == kv + qo + meta + partial


def test_algorithmic_bytes_b1_workload():
    # the B1 step the roofline is taken on: the last of 20 steps (32768 + 20 tokens), 256 tasks
    total, kv = bench.algorithmic_bytes([32788], 256)
    assert kv == 4096 * 32788 and total == 135394324       # the figure in the committed profiles


def test_read_traffic_requires_the_current_kernel(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "PROFILES", str(tmp_path))
    assert bench.read_traffic("b1") is None               # no summary
    body = "- hbm_bytes_per_dispatch: 123456\n- kernel_source_sha256: {}\n"
    (tmp_path / "counters_split_kernel_b1.md").write_text(body.format("0" * 16))
    assert bench.read_traffic("b1") is None               # taken on another kernel source
    (tmp_path / "counters_split_kernel_b1.md").write_text(body.format(bench.kernel_hash()))
    assert bench.read_traffic("b1") == 123456.0


def test_committed_profiles_parse():
    """The committed counter summaries carry the fields bench.py reads; when they were taken
    on another kernel source the test is skipped (bench.py then reports traffic as null)."""
    import pytest
    for w in ("b1", "b8_bimodal"):
        text = open(os.path.join(bench.PROFILES, f"counters_split_kernel_{w}.md")).read()
        assert "- hbm_bytes_per_dispatch: " in text and "- kernel_source_sha256: " in text
        if bench.read_traffic(w) is None:
            pytest.skip("profiles were taken on another kernel source")


def test_head_pair_report():
    assert bench.head_pairs(32, 8, 512) and not bench.head_pairs(32, 8, 256)
    assert not bench.head_pairs(32, 4, 512) and not bench.head_pairs(32, 32, 1024)


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2 and "one MI355X" in r.stderr
    assert np.isfinite(bench.HBM_PEAK_GBS) and bench.HBM_PEAK_GBS == 8000.0
