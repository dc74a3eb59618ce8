"""Host-side checks of bench.py: the one-GPU contract and the counter
summaries it reads its HBM traffic from (no GPU needed)."""
import glob
import json
import os
import re
import subprocess
import sys

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120, cwd=ROOT)
    assert r.returncode != 0
    assert "one GPU only" in r.stderr
    assert r.stdout.strip() == ""            # no JSON line for a run that did not happen


def _blocks():
    for path in sorted(glob.glob(os.path.join(ROOT, "profiles", "pmc_*.md"))):
        m = re.search(r"```json\n(.*?)\n```", open(path).read(), re.S)
        assert m, f"{path}: no JSON block"
        yield path, json.loads(m.group(1))


def test_counter_summaries_are_consistent():
    """Each summary's bytes follow from its counters and the copy calibration,
    and it names a kernel family and a workload that bench.py measures."""
    paths = []
    for path, d in _blocks():
        paths.append(path)
        key, workload = re.match(r"pmc_(.+?)_(.+)\.md$", os.path.basename(path)).groups()
        assert key in bench.KERNELS, path
        assert d["workload"] == workload, path
        cal = d["copy_calibration"]
        # the scales are the copy's bytes over the counters' bytes
        assert abs(cal["fetch_scale"] - cal["bytes_read"] / (cal["fetch_kib"] * 1024)) < 1e-3
        assert abs(cal["write_scale"] - cal["bytes_written"] / (cal["write_kib"] * 1024)) < 1e-3
        # bytes per launch use the unrounded scales
        rd = d["fetch_kib_per_dispatch"] * cal["bytes_read"] / cal["fetch_kib"]
        wr = d["write_kib_per_dispatch"] * cal["bytes_written"] / cal["write_kib"]
        assert abs(d["hbm_bytes_read_per_launch"] - rd) <= 1e-6 * rd + 1024, path
        assert abs(d["hbm_bytes_written_per_launch"] - wr) <= 1e-6 * wr + 1024, path
        # each figure is rounded from the unrounded bytes on its own
        assert abs(d["hbm_bytes_per_launch"] - d["hbm_bytes_read_per_launch"]
                   - d["hbm_bytes_written_per_launch"]) <= 1, path
        # X read once and the labels written: n (4M + 4) bytes
        m = re.search(r"n = ([\d,]+), M = (\d+)", open(path).read())
        n, M = int(m.group(1).replace(",", "")), int(m.group(2))
        assert d["algorithmic_bytes_per_launch"] == n * (4 * M + 4), path
        # traffic at least the algorithmic bytes (X crosses HBM at least once)
        assert d["hbm_bytes_per_launch"] >= 0.99 * d["algorithmic_bytes_per_launch"], path
    assert paths, "no counter summaries under profiles/"


def test_traffic_is_withheld_when_the_sources_changed(tmp_path, monkeypatch):
    """bench.py reports a summary's traffic only while the kernel sources
    still hash to the summary's `sources_sha256`."""
    path, d = next(_blocks())
    key, workload = re.match(r"pmc_(.+?)_(.+)\.md$", os.path.basename(path)).groups()
    monkeypatch.setattr(bench, "PROFILES", str(tmp_path))
    target = tmp_path / os.path.basename(path)
    d_now = dict(d, sources_sha256=bench.sources_sha256(key))
    target.write_text("```json\n" + json.dumps(d_now) + "\n```\n")
    assert bench._traffic(key, workload) == d["hbm_bytes_per_launch"]
    target.write_text("```json\n" + json.dumps(dict(d, sources_sha256="0" * 64)) + "\n```\n")
    assert bench._traffic(key, workload) is None
