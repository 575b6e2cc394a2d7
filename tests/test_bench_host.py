"""Host-side logic of bench.py (no GPU): kernel-name classification of the
rocprofv3 traces, the algorithmic byte counts behind the roofline figures, the
split of a trace by workload, and the one-GPU guard."""
import os
import subprocess
import sys

import pytest
import torch

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402

P = "void q2d::(anonymous namespace)::"


@pytest.mark.parametrize("name,kind", [
    (P + "gemm_fp4_persistent_kernel<true, false, 0, 0, false>(q2d::GemmArgs, int, int, q2d::GroupedArgs)", "gemm_fp4"),
    (P + "gemm_fp4_persistent_kernel<false, true, 0, 3, false>(q2d::GemmArgs, int, int, q2d::GroupedArgs)", "gemm_fp4"),
    (P + "gemm_fp4_persistent_kernel<true, false, 1, 0, false>(q2d::GemmArgs, int, int, q2d::GroupedArgs)",
     "gemm_fp4_grouped"),
    (P + "gemm_fp4_persistent_kernel<false, false, 2, 0, false>(q2d::GemmArgs, int, int, q2d::GroupedArgs)",
     "gemm_fp4_grouped_k"),
    (P + "gemm_fp4_persistent_kernel<false, false, 0, 1, true>(q2d::GemmArgs, int, int, q2d::GroupedArgs)",
     "gemm_fp4_yq"),
    (P + "gemm_fp4_persistent_kernel<false, false, 0, 0, true, false>(q2d::GemmArgs, int, int, q2d::GroupedArgs)",
     "gemm_fp4_yq"),
    (P + "gemm_fp4_persistent_kernel<false, false, 0, 0, true, true>(q2d::GemmArgs, int, int, q2d::GroupedArgs)",
     "gemm_fp4_dxq"),
    (P + "gemm_fp8_256_kernel<true, false>(q2d::GemmArgs, int, int)", "gemm_fp8"),
    (P + "gemm_kernel<0, true>(q2d::GemmArgs, long, long)", "gemm_fp4"),
    (P + "gemm_kernel<1, false>(q2d::GemmArgs, long, long)", "gemm_fp8"),
    (P + "fp4_quantize_kernel<unsigned short, true, false, true, false, 2, false>(q2d::QuantArgs)", "quant_fp4"),
    (P + "fp4_quantize_kernel<float, true, true, true, true, 1, false>(q2d::QuantArgs)", "quant_fp4_grouped"),
    (P + "fp4_quantize_kernel<unsigned short, true, false, true, false, 2, true>(q2d::QuantArgs)", "quant_fp4_1d"),
    (P + "mxfp8_quantize_kernel<false, true>(q2d::QuantArgs)", "quant_mxfp8"),
    ("void at::native::vectorized_elementwise_kernel<4, at::native::FillFunctor<float>>(int, float, float)", None),
])
def test_kind_of(name, kind):
    assert bench.kind_of(name) == kind


def test_every_kind_has_peak_kernel_and_source():
    for k in bench.KIND_PEAK:
        assert k in bench.KIND_KERNEL and k in bench.KIND_SOURCES


def test_byte_counts():
    t = torch.empty((64, 96), dtype=torch.bfloat16)
    n = 64 * 96
    assert bench.quant_bytes(t) == n * 2 + n + n / 1024
    assert bench.quant_bytes(t, "fp4_1d") == n * 2 + n + 2 * n / 32
    assert bench.quant_bytes(t, "mxfp8") == n * 2 + 2 * n + 2 * n / 32
    # A [M, K], B [N, K] FP4 codes with 2D scales, bf16 C [M, N]
    M, N, K = 256, 128, 512
    assert bench.gemm_bytes(M * K, N * K, M * N * 2) == (M * K + N * K) * (0.5 + 1 / 1024) + M * N * 2
    assert bench.gemm_bytes(M * K, N * K, 0, "fp4", True, False) == M * K * (0.5 + 1 / 32) + N * K * (0.5 + 1 / 1024)


def test_phase_owners():
    assert bench.phase_owners(5, [("a", 2), ("b", 3)]) == ["a", "a", "b", "b", "b"]
    with pytest.raises(ValueError):
        bench.phase_owners(4, [("a", 2), ("b", 3)])


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2 and "one GPU" in r.stderr
