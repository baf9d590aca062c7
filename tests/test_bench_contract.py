"""CPU checks of bench.py's command-line contract (no GPU involved): more than one GPU is refused
with a JSON message before anything touches a device, and the kernel labels the benchmark
reports follow the library's routing by batch size."""
from __future__ import annotations

import json
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def test_more_than_one_gpu_is_refused():
    res = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2", "--steps", "1"],
                         capture_output=True, text=True, timeout=120, cwd=ROOT)
    assert res.returncode == 2
    line = json.loads(res.stdout.strip().splitlines()[-1])
    assert line["n_gpus"] == 2 and "one GPU" in line["error"]


def test_kernel_labels_follow_batch_routing():
    assert bench.kernel_label("W2", 1).startswith("k_gemm_valu<W2,M=1>")
    assert bench.kernel_label("W2", 2).startswith("k_gemm_valu<W2,M=2>")
    assert bench.kernel_label("W3", 2).startswith("k_gemm_valu<W3,M=4>")    # no two-row kernel for 2^13 codebooks
    assert bench.kernel_label("W2", 3).startswith("k_gemm_valu<W2,M=4>")
    assert bench.kernel_label("W2", 8).startswith("k_gemm_valu<W2,M=8>")
    assert bench.kernel_label("W2", 16).startswith("k_gemm_valu<W2,M=16>")
    assert bench.kernel_label("W2", 17).startswith("k_gemm_prefill<W2>")
    # batches 9..16 go to the prefill kernel from 120 * 2^20 weights (the library's routing bound)
    assert bench.kernel_label("W2", 12, 24576, 4096).startswith("k_gemm_valu<W2,M=16>")   # 96 * 2^20
    assert bench.kernel_label("W2", 12, 32768, 4096).startswith("k_gemm_prefill<W2>")     # 128 * 2^20
    assert bench.kernel_label("W2", 16, 51200, 5120).startswith("k_gemm_prefill<W2>")
    assert bench.kernel_label("W2", 8, 51200, 5120).startswith("k_gemm_valu<W2,M=8>")
    assert bench.kernel_label("V4", 1).startswith("k_gemm_rowvec<V4,MB=1>")
    assert bench.kernel_label("V16", 5).startswith("k_gemm_rowvec<V16,MB=8>")


def test_peaks_are_the_published_figures():
    assert bench.HBM_PEAK_GBS == 8000.0
    assert bench.MFMA_F16_PEAK_TFS == 2500.0
