"""CPU checks of bench.py's host logic: the one-GPU refusal and the HBM
traffic record, which is used only for the library file it was taken with
or while the kernel sources it was taken on are unchanged."""

import hashlib
import json
import os
import subprocess
import sys

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_traffic_record_follows_its_sources(tmp_path, monkeypatch):
    src = tmp_path / "k.hip"
    src.write_text("kernel source\n")
    rec = {"sources": {"k.hip": hashlib.sha256(src.read_bytes()).hexdigest()},
           "workloads": {"cfg3": {"P.gemm1_swiglu": {"hbm_bytes": 12345}}}}
    (tmp_path / "profiles").mkdir()
    (tmp_path / "profiles" / "hbm_traffic.json").write_text(json.dumps(rec))
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    assert bench.recorded_traffic(3, 0, "gemm1_swiglu") == 12345
    assert bench.recorded_traffic(3, 1, "gemm1_swiglu") is None  # no record for D
    assert bench.recorded_traffic(2, 0, "gemm1_swiglu") is None  # nor for another workload
    src.write_text("kernel source, changed\n")
    assert bench.recorded_traffic(3, 0, "gemm1_swiglu") is None
    src.unlink()
    assert bench.recorded_traffic(3, 0, "gemm1_swiglu") is None


def test_traffic_record_follows_the_profiled_library(tmp_path, monkeypatch):
    src = tmp_path / "k.hip"
    src.write_text("kernel source\n")
    lib = tmp_path / "lib.so"
    lib.write_bytes(b"\x7fELF profiled build")
    rec = {"sources": {"k.hip": hashlib.sha256(b"another source\n").hexdigest()},
           "library_sha256": hashlib.sha256(lib.read_bytes()).hexdigest(),
           "workloads": {"cfg3": {"P.gemm1_swiglu": {"hbm_bytes": 777}}}}
    (tmp_path / "profiles").mkdir()
    (tmp_path / "profiles" / "hbm_traffic.json").write_text(json.dumps(rec))
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    # the sources differ, the library is the profiled one
    assert bench.recorded_traffic(3, 0, "gemm1_swiglu", str(lib)) == 777
    assert bench.recorded_traffic(3, 0, "gemm1_swiglu") is None
    lib.write_bytes(b"\x7fELF another build")
    assert bench.recorded_traffic(3, 0, "gemm1_swiglu", str(lib)) is None
    assert bench.recorded_traffic(3, 0, "gemm1_swiglu", str(tmp_path / "missing.so")) is None
