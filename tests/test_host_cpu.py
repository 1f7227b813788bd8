"""CPU checks of host-side logic: bench.py's single-GPU guard and traffic-record matching,
and the binding's refusal to run without the built library (no fallback path)."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)


def test_bench_refuses_more_than_one_gpu():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_traffic_record_must_match_kernels_and_launch(tmp_path, monkeypatch):
    import bench
    h = bench.score_source_hash()
    assert len(h) == 64 and h == bench.score_source_hash()
    rec = {"source_sha256": h, "layers_per_call": 32, "hbm_bytes_per_call": 123}
    (tmp_path / "profiles").mkdir()
    (tmp_path / "profiles" / "score_traffic_cx.json").write_text(json.dumps(rec))
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    monkeypatch.setattr(bench, "score_source_hash", lambda: h)
    assert bench.measured_traffic("cx", False, 32) == 123
    assert bench.measured_traffic("cx", False, 1) is None          # other launch shape
    rec["source_sha256"] = "0" * 64
    (tmp_path / "profiles" / "score_traffic_cx.json").write_text(json.dumps(rec))
    assert bench.measured_traffic("cx", False, 32) is None         # kernels changed
    assert bench.measured_traffic("cy", False, 32) is None         # no record


def test_missing_library_raises(monkeypatch):
    from paper_2609_33334_amd import _lib
    monkeypatch.setattr(_lib, "_lib", None)
    monkeypatch.setattr(_lib, "LIB_PATH", os.path.join(ROOT, "no_such_dir", "libdge.so"))
    with pytest.raises(RuntimeError, match="no fallback"):
        _lib.lib()
