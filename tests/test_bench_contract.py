"""bench.py pieces that need no GPU: the one-GPU guard, the algorithmic
bytes of a simulation, and the traffic record (HBM bytes per launch from a
committed counter summary, reported only while the kernel sources hash to
the recorded value)."""
import hashlib
import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402
from paper_2607_11262_amd.gen.graph import DATA, GLOAD, GSTORE, GraphBuilder  # noqa: E402


def test_more_than_one_gpu_is_refused(monkeypatch, capsys):
    monkeypatch.setattr(sys, "argv", ["bench.py", "--gpus", "4"])
    assert bench.main() == 2
    assert "one GPU" in capsys.readouterr().err


def test_algorithmic_bytes():
    b = GraphBuilder()
    b.kernel(4, 0)
    b.cta()
    a = b.node(GLOAD, 256, 1)
    s = b.node(GSTORE, 256, 1)
    b.edge(a, s, DATA)
    g = b.build("two")
    assert bench.alg_bytes_per_sim(g) == 16 * 2 + 4 * 1 + 16


def _sources_hash():
    h = hashlib.sha256()
    for name in bench.KERNEL_SOURCES:
        with open(os.path.join(ROOT, "paper_2607_11262_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def _record(tmp_path, sha, launches=4):
    p = tmp_path / "summary.md"
    p.write_text(f"text\n    traffic-record: sha256={sha} launches={launches} fetch_kib=1000 write_kib=3000 "
                 f"fetch_factor=2.0000 write_factor=1.0000\n")
    return str(p)


def test_traffic_record_read_while_sources_match(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "PROFILE", _record(tmp_path, _sources_hash()))
    assert bench.recorded_traffic(4) == pytest.approx((1000 * 1024 * 2.0 + 3000 * 1024 * 1.0) / 4)


def test_traffic_record_ignored_for_other_sources_or_launches(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "PROFILE", _record(tmp_path, "0" * 64))
    assert bench.recorded_traffic(4) is None
    monkeypatch.setattr(bench, "PROFILE", _record(tmp_path, _sources_hash()))
    assert bench.recorded_traffic(5) is None
    monkeypatch.setattr(bench, "PROFILE", str(tmp_path / "missing.md"))
    assert bench.recorded_traffic(4) is None

