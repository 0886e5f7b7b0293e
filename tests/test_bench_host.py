"""Host-side logic of bench.py (no GPU): the one-GPU contract and the rule that
the gate/up HBM traffic in the JSON line comes only from a counter summary
taken on the current GEMM source."""
import os
import subprocess
import sys

import pytest

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_exits_with_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU only" in r.stderr
    assert r.stdout.strip() == ""  # no JSON line for an unsupported run


def _summary(tmp_path, wid, text):
    d = tmp_path / "profiles"
    d.mkdir(exist_ok=True)
    (d / bench.TRAFFIC_FILES[wid]).write_text(text)


@pytest.mark.parametrize("wid", sorted(bench.TRAFFIC_FILES))
def test_traffic_read_only_for_matching_source(tmp_path, monkeypatch, wid):
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    monkeypatch.setattr(bench, "kernel_source_hash", lambda: "00ff00ff00ff00ff")
    assert bench.load_traffic(wid) is None  # no summary
    body = "command:\n    rocprofv3 --pmc FETCH_SIZE ...\nhbm_bytes_per_launch: 123456789\n"
    _summary(tmp_path, wid, body + "kernel_source_hash: 00ff00ff00ff00ff\n")
    assert bench.load_traffic(wid) == 123456789
    _summary(tmp_path, wid, body + "kernel_source_hash: 1111111111111111\n")
    assert bench.load_traffic(wid) is None  # taken on another source: null
    _summary(tmp_path, wid, "kernel_source_hash: 00ff00ff00ff00ff\nhbm_bytes_per_launch: n/a\n")
    assert bench.load_traffic(wid) is None


def test_no_traffic_for_workloads_without_summary(monkeypatch):
    for wid in (1, 3, 5):
        assert wid not in bench.TRAFFIC_FILES
        assert bench.load_traffic(wid) is None


# gate/up algorithmic bytes per launch: packed rows read, both weight matrices
# read, activations written (bf16); the committed counters must not read below it
ALGO_BYTES = {2: 4408 * 1536 * 2 + 2 * 1536 * 8960 * 2 + 4408 * 8960 * 2,
              4: 5122 * 3584 * 2 + 2 * 3584 * 18944 * 2 + 5122 * 18944 * 2}


@pytest.mark.parametrize("wid", sorted(bench.TRAFFIC_FILES))
def test_committed_traffic_summary_parses(monkeypatch, wid):
    path = os.path.join(ROOT, "profiles", bench.TRAFFIC_FILES[wid])
    with open(path) as f:
        lines = [ln for ln in f if ln.startswith("kernel_source_hash:")]
    assert len(lines) == 1
    declared = lines[0].split(":", 1)[1].strip()
    monkeypatch.setattr(bench, "kernel_source_hash", lambda: declared)
    got = bench.load_traffic(wid)
    assert isinstance(got, int)
    assert got >= ALGO_BYTES[wid]
