"""CPU checks of bench.py's host logic: the single-GPU contract and the
reduction of rocprofv3 counter runs into HBM bytes per GEMM launch."""

import csv
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def test_bench_refuses_several_gpus():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout.strip() == ""


def _write_counters(path, rows):
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Kernel_Name", "Counter_Value"])
        w.writeheader()
        for name, value in rows:
            w.writerow({"Kernel_Name": name, "Counter_Value": value})


def test_reduce_counters_scales_each_counter_by_the_copy_probe(tmp_path):
    # a 256 MiB probe whose FETCH_SIZE reads half its bytes (factor 2) and
    # whose WRITE_SIZE reads them exactly (factor 1); three GEMM dispatches
    g = f"void qwam::{bench.GEMM_KERNEL}(unsigned char const*, ...)"
    c = f"{bench.COPY_KERNEL}HIP_vector_type<unsigned int, 4u> const*, ...)"
    torch_copy = "void at::native::vectorized_elementwise_kernel<4, copy_kernel(...)"
    fetch, write = tmp_path / "f.csv", tmp_path / "w.csv"
    _write_counters(fetch, [(g, 1000.0), (c, 131072.0), (torch_copy, 7.0), (g, 1100.0), (g, 900.0)])
    _write_counters(write, [(c, 262144.0), (g, 500.0), (g, 500.0), (g, 500.0)])
    rec = bench.reduce_counters(str(fetch), str(write), 256)
    assert rec["fetch_factor"] == pytest.approx(2.0)
    assert rec["write_factor"] == pytest.approx(1.0)
    assert rec["fetch_launches"] == 3 and rec["write_launches"] == 3
    assert rec["bytes_per_launch"] == (1000 * 2 + 500 * 1) * 1024
    assert rec["gemm_source_sha256_16"] == bench.source_hash(bench.GEMM_SRCS)


def test_reduce_counters_requires_both_kernels(tmp_path):
    g = f"void qwam::{bench.GEMM_KERNEL}(...)"
    fetch, write = tmp_path / "f.csv", tmp_path / "w.csv"
    _write_counters(fetch, [(g, 1000.0)])
    _write_counters(write, [(g, 500.0)])
    with pytest.raises(SystemExit):
        bench.reduce_counters(str(fetch), str(write), 256)
