"""Host-side checks of bench.py (no GPU): the one-GPU contract, the arithmetic that turns rocprofv3 CSVs into
the committed summaries, and the recycled-block count against the oracle's scan of later steps."""
import csv
import os
import subprocess
import sys

import numpy as np
import pytest

from oracle import paged as OP

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_more_than_one_gpu_is_refused():
    res = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                         text=True, timeout=120)
    assert res.returncode == 2
    assert "one GPU" in res.stderr
    assert res.stdout == ""


def write_counters(path, rows):
    os.makedirs(path, exist_ok=True)
    with open(os.path.join(path, "x_counter_collection.csv"), "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Kernel_Name", "Counter_Value"])
        w.writeheader()
        for name, value in rows:
            w.writerow({"Kernel_Name": name, "Counter_Value": value})


def test_traffic_summary_arithmetic(tmp_path):
    """FETCH_SIZE and WRITE_SIZE per dispatch of the named kernel (mean over its dispatches, others ignored),
    each scaled so that a plain copy of known size reads its true bytes."""
    k = "decode_attn_wide_kernel<1>"
    write_counters(tmp_path / "f", [(k, 100.0), (k, 300.0), ("other", 9e9)])
    write_counters(tmp_path / "w", [(k, 40.0), ("other", 1.0)])
    write_counters(tmp_path / "cf", [("__amd_rocclr_copyBuffer", 512.0)])  # a 1 MiB copy: fetch under-reads 2x
    write_counters(tmp_path / "cw", [("__amd_rocclr_copyBuffer", 1024.0)])
    text = bench.summarize_pmc("c3", k, str(tmp_path / "f"), str(tmp_path / "w"), str(tmp_path / "cf"),
                               str(tmp_path / "cw"), 1, 1000)
    fields = dict(line.split(": ", 1) for line in text.splitlines() if not line.startswith("#"))
    assert float(fields["fetch_kib_per_dispatch"]) == 200.0
    assert float(fields["write_kib_per_dispatch"]) == 40.0
    assert float(fields["fetch_scale"]) == 2.0 and float(fields["write_scale"]) == 1.0
    assert float(fields["traffic_bytes_per_launch"]) == (200.0 * 2 + 40.0) * 1024
    assert fields["kernel_source_sha256_16"] == bench.kernel_source_hash()


def test_committed_traffic_needs_the_current_kernel(tmp_path, monkeypatch):
    """The bench reports the committed traffic only while the summary's kernel hash matches kernels.hip."""
    prof = tmp_path / "profiles"
    prof.mkdir()
    good = f"traffic_bytes_per_launch: 123\nkernel_source_sha256_16: {bench.kernel_source_hash()}\n"
    (prof / "decode_attn_c3_traffic.txt").write_text(good)
    (prof / "decode_attn_c5_traffic.txt").write_text("traffic_bytes_per_launch: 5\nkernel_source_sha256_16: 0\n")
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    assert bench.committed_traffic("c3") == 123.0
    assert bench.committed_traffic("c5") is None
    assert bench.committed_traffic("c1") is None


def test_recycled_block_count_matches_the_oracle():
    """bench.recycled_blocks (closed form, per step) equals a count from the oracle's freeable blocks on a
    small layout decoded to 60 outputs."""
    seg0 = np.array([[4, 40, 1, 0], [0, 25, 0, 0]], dtype=np.int32)
    pol = np.array([[8, 3, 2, 6, 1], [5, 0, 0, 4, 0]], dtype=np.int32)
    got = bench.recycled_blocks(seg0, pol, block_size=4, n_outputs=60)
    peak = 0
    for j in range(1, 61):
        held = 0
        for b in range(2):
            row = [int(x) for x in seg0[b]]
            row[3] = j
            blocks = -(-sum(row) // 4)
            held += blocks - len(OP.freeable_blocks(row, pol[b], 4))
        peak = max(peak, held)
    assert got["peak_blocks"] == peak
    assert got["blocks_without_freeing"] == sum(-(-(int(seg0[b, :3].sum()) + 60) // 4) for b in range(2))


def test_kernel_hash_ignores_comments_only():
    """The traffic gate's hash changes with the kernel code, not with its comments or layout."""
    a = "int f(int x) { return x + 1; } // one\n/* two\n lines */ int g;"
    b = "int f(int x)  {\n  return x + 1;\n}\n// other words\nint g;"
    c = "int f(int x) { return x + 2; } int g;"
    assert bench.kernel_code_text(a) == bench.kernel_code_text(b)
    assert bench.kernel_code_text(a) != bench.kernel_code_text(c)
