"""Host-side checks of the benchmark's bookkeeping (CPU only): the ceilings
it prices each arithmetic at, the bound it picks, and the epoch order it
times."""
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import bench  # noqa: E402
import pmlp_workloads as wl  # noqa: E402


def test_ceilings_follow_the_reported_arithmetic():
    import paper_2206_08369_amd as pm
    assert bench.mfma_peak(pm.PMLP_ARITH_FP32) == bench.PEAK_FP32_MFMA
    assert bench.mfma_peak(pm.PMLP_ARITH_X3) == bench.PEAK_BF16_MFMA / 6
    assert bench.mfma_peak(pm.PMLP_ARITH_BF16) == bench.PEAK_BF16_MFMA
    assert bench.mfma_peak(pm.PMLP_ARITH_NONE) is None


def test_bounds():
    w = wl.WORKLOADS["w10k_f100"]
    N, M = w.N, w.M
    x3 = bench.PEAK_BF16_MFMA / 6
    # at F = 100, B = 256 both products sit below the 52 flop/B ridge of the
    # three-piece ceiling (36 and 29 flop/B) but above the fp32 ridge
    for k in ("gemm_fwd", "bwd_fused"):
        bound, nbytes, flops = bench.kernel_work(k, w.B, w.F, N, M, w.O)
        assert 19.7 < flops / nbytes < 52
        assert bench.roofline_bound(bound, nbytes, flops, x3) == "hbm"
        assert bench.roofline_bound(bound, nbytes, flops, bench.PEAK_FP32_MFMA) == "mfma"
        assert bench.roofline_bound(bound, nbytes, flops, None) == "hbm"
    # bandwidth kernels stay bandwidth-bound whatever the ceiling
    bound, nbytes, flops = bench.kernel_work("m3_fwd", w.B, w.F, N, M, w.O)
    assert bench.roofline_bound(bound, nbytes, flops, 1e6) == "hbm"


def test_epochs_end_with_their_partial_batch():
    for name, last in (("w10k_f100", 16), ("w10k_f1000", 672), ("w10k_f32_o10", 16),
                       ("w60_f10", 8)):
        w = wl.WORKLOADS[name]
        b = bench.epoch_batches(w)
        assert b[-1][1] == last and sum(n for _, n in b) == w.S
        assert all(n == w.B for _, n in b[:-1])


def test_every_reported_kernel_has_a_source_file():
    """Traffic entries are tied to the source file that defines their kernel;
    every name the library can report (its variant notes) must resolve."""
    import re
    csrc = os.path.join(ROOT, "paper_2206_08369_amd", "csrc")
    names = set()
    for f in os.listdir(csrc):
        if f.endswith(".hip"):
            names |= set(re.findall(r'note_variant\("(\w+)"', open(os.path.join(csrc, f)).read()))
    assert {"k_fwd_x3", "k_bwd_x3", "k_gemm_x3", "k_gemm_bf", "k_gemm_nt"} <= names
    for n in names:
        src = bench.kernel_source(n)
        assert src is not None, n
        assert re.search(r"\bvoid\s+%s\s*\(" % bench.VARIANT_KERNEL.get(n, n),
                         open(os.path.join(csrc, src)).read()), n
    assert bench.kernel_source("k_gemm_x3") == bench.kernel_source("k_gemm_bf") == "k_gemm_bf16.hip"
    assert bench.kernel_source("k_bwd_x3<6, 2, 2, 512, true>") == "k_lds.hip"
    # the digest changes with the kernel's own file, not with other kernels' files
    assert bench.kernel_source_digest("k_m3_fwd") != bench.kernel_source_digest("k_fwd_x3")


def test_profile_roles_read_the_epilogue_argument():
    import bench_profiles as bp
    assert bp.role_of("k_gemm_bf<4, 2, 2, 4, 16, false, 0, true>", "fp32") == "gemm_fwd"
    assert bp.role_of("k_gemm_bf<4, 2, 2, 4, 32, true, 1, false>", "bf16") == "gemm_bwd"
    assert bp.role_of("k_gemm_bf<4, 2, 2, 4, 32, false, 2, false>", "bf16") == "gemm_grad"
    assert bp.role_of("k_gemm_nt<4, 2, 1>", "fp32") == "gemm_bwd"
    assert bp.role_of("k_bwd_x3<6, 2, 2, 512, true>", "fp32") == "bwd_fused"
