"""Host-side checks of the benchmark's roofline bookkeeping (CPU only): which
kernels it prices at the three-piece ceiling, and the bound it picks."""
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import bench  # noqa: E402
import pmlp_workloads as wl  # noqa: E402


def test_three_piece_kernels_of_each_workload():
    # the kernels the library launches for each workload, as its kernel
    # traces name them: k_fwd_x3 / k_bwd_x3 for F = 100 and F = 50 at 256 and
    # 128 samples; k_fwd_lds_ring / k_bwd_mf at 32 samples; the generic or
    # bf16 GEMMs at F = 1000
    expect = {"w10k_f100": (True, True), "paper_10k": (True, True), "w1k_f50": (True, True),
              "w10k_f32_o10": (False, False), "w10k_f1000": (False, False),
              "w60_f10": (False, False)}
    for name, (fwd, bwd) in expect.items():
        w = wl.WORKLOADS[name]
        assert bench.three_piece("gemm_fwd", w.B, w.F, w.O) == fwd, name
        assert bench.three_piece("bwd_fused", w.B, w.F, w.O) == bwd, name


def test_ceilings_and_bounds():
    w = wl.WORKLOADS["w10k_f100"]
    N, M = w.N, w.M
    assert bench.mfma_peak("bwd_fused", w.B, w.F, w.O) == bench.PEAK_BF16_MFMA / 6
    assert bench.mfma_peak("bwd_fused", 32, w.F, w.O) == bench.PEAK_FP32_MFMA
    assert bench.mfma_peak("gemm_fwd", w.B, w.F, w.O, "bf16") == bench.PEAK_BF16_MFMA
    # at F = 100, B = 256 both products sit below the 52 flop/B ridge of the
    # three-piece ceiling (36 and 29 flop/B) but above the fp32 ridge
    for k in ("gemm_fwd", "bwd_fused"):
        bound, nbytes, flops = bench.kernel_work(k, w.B, w.F, N, M, w.O)
        assert 19.7 < flops / nbytes < 52
        assert bench.roofline_bound(bound, nbytes, flops,
                                    bench.mfma_peak(k, w.B, w.F, w.O)) == "hbm"
        assert bench.roofline_bound(bound, nbytes, flops, bench.PEAK_FP32_MFMA) == "mfma"
    # bandwidth kernels stay bandwidth-bound whatever the ceiling
    bound, nbytes, flops = bench.kernel_work("m3_fwd", w.B, w.F, N, M, w.O)
    assert bench.roofline_bound(bound, nbytes, flops, 1e6) == "hbm"


def test_padded_batch():
    assert [bench.padded_batch(b) for b in (1, 16, 17, 100, 128, 129, 256)] == \
        [16, 16, 32, 128, 128, 256, 256]
    assert bench.padded_batch(257) is None
