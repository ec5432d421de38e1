"""Benchmark: packed ParallelMLPs SGD training steps on one MI355X.

One step = one batch through the whole hot path (batch packing, the
input-layer GEMM, fused activation + M3 forward, per-model softmax
cross-entropy, M3 backward with the W2 update, and the dW1 GEMM with the
W1 update).  Inputs are seeded synthetic data shaped like the paper's
simulated workloads, resident in GPU memory before timing; weights start
from the library's seeded initialisation.

Prints ONE JSON line with the throughput in model-samples trained per
second, the roofline position of the dominant kernel (per-kernel times
from HIP events recorded on the library's stream inside the timed region)
and the CPU oracle's rate on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

import pmlp_workloads as wl  # noqa: E402

METRIC = "model-samples trained/sec (fwd+bwd+SGD) + % MFMA/HBM roofline, 10k MLPs"
PEAK_HBM_GBS = 8000.0          # MI355X HBM3E, GB/s
PEAK_FP32_MFMA = 157.3         # TFLOP/s, dense fp32 matrix
PEAK_BF16_MFMA = 2500.0        # TFLOP/s, dense bf16 matrix


def kernel_work(name, B, F, N, M, O, precision="fp32"):
    """(bound, algorithmic bytes, algorithmic flops) of one launch.

    Bytes count each tensor the kernel must read or write once, at the width
    the path stores it: fp32, except in the bf16 mode the batch copies, the
    bf16 copy of W1 (read by the input-to-hidden product, rewritten by the
    update) and dZ (written by the M3 backward, read by the dW1 product);
    flops count multiply-adds as two operations."""
    f4 = 4.0
    bf = precision == "bf16"
    fx = 2.0 if bf else 4.0      # bytes per element of the batch copy
    if name == "gemm_fwd":       # Z = X W1^T: read W1 (bf16 copy in bf16 mode), X; write Z
        return "mfma", (2.0 if bf else f4) * N * F + fx * B * F + f4 * N * B, 2.0 * B * F * N
    if name == "gemm_bwd":       # W1 -= lr dZ^T X: read dZ, X; read+write W1 (+ its bf16 copy)
        return ("mfma", (2.0 if bf else f4) * N * B + fx * B * F + 2 * f4 * N * F
                + (2.0 * N * F if bf else 0.0), 2.0 * B * F * N)
    if name == "m3_fwd":         # read Z, W2; write logits
        return "hbm", f4 * (N * B + O * N + B * M * O), 2.0 * B * O * N
    if name == "m3_bwd":         # read Z, G, W2; write dZ (bf16 in bf16 mode), W2
        return ("hbm", f4 * N * B + (2.0 if bf else f4) * N * B + f4 * (2 * O * N + B * M * O),
                4.0 * B * O * N)
    if name == "bwd_fused":      # read Z, G, X; read+write W1 and W2 (dZ stays in registers)
        return ("mfma", f4 * (N * B + B * M * O + B * F + 2 * N * F + 2 * O * N),
                2.0 * B * F * N + 4.0 * B * O * N)
    if name == "ce":             # read logits, y; write G, loss
        return "hbm", f4 * (2 * B * M * O + B + M), 0.0
    if name == "pack_x":         # read X; write two padded copies
        return "hbm", f4 * B * F + 2 * fx * B * F, 0.0
    return "hbm", 0.0, 0.0


LDS_BYTES = 160 * 1024        # per workgroup


def padded_batch(B):
    """Batch width of the LDS-resident kernels: 16, 32, 64, 128 or 256."""
    return next((b for b in (16, 32, 64, 128, 256) if B <= b), None)


def three_piece(name, B, F, O):
    """True where the fp32 path runs the kernel's matrix products as six
    bf16 products of three-piece operand splits (batches of 128 and 256
    samples): the input-layer forward when its three LDS planes fit, the
    fused backward for F4 = 52 or 100 and O = 2."""
    bp, f4 = padded_batch(B), (F + 3) // 4 * 4
    if bp not in (128, 256):
        return False
    if name == "gemm_fwd":
        lds = 3 * bp * (f4 // 32) * 64 + bp * ((f4 % 32) // 4) * 16
        return 32 <= f4 <= 140 and bp * f4 * 4 <= LDS_BYTES and lds <= LDS_BYTES
    if name == "bwd_fused":
        return O == 2 and f4 in (52, 100)
    return False


def mfma_peak(name, B, F, O, precision="fp32"):
    """Matrix-core ceiling of one kernel in TFLOP/s of its own arithmetic:
    the bf16 peak in the bf16 mode; in the fp32 path the fp32 peak, or a
    sixth of the bf16 peak where each fp32 multiply-add is six bf16 ones."""
    if precision == "bf16":
        return PEAK_BF16_MFMA
    return PEAK_BF16_MFMA / 6.0 if three_piece(name, B, F, O) else PEAK_FP32_MFMA


def roofline_bound(bound, nbytes, flops, peak_tflops):
    """A matrix-core kernel is compute-bound only when its arithmetic
    intensity (algorithmic flops per algorithmic byte) is above the ridge
    point of its matrix-core ceiling (peak flops / peak HBM bandwidth);
    below it the HBM roofline bounds it."""
    if bound != "mfma" or not nbytes:
        return bound
    ridge = peak_tflops * 1e12 / (PEAK_HBM_GBS * 1e9)
    return "mfma" if flops / nbytes >= ridge else "hbm"


def traffic_key(kernel: str, workload: str, precision: str) -> str:
    return "%s/%s%s" % (kernel, workload, "" if precision == "fp32" else "+" + precision)


def load_traffic(kernel: str, workload: str, precision: str = "fp32"):
    """HBM bytes per launch from committed rocprofv3 counter summaries, if
    they were taken on the current kernel source; otherwise None."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    try:
        table = json.load(open(path))
    except ValueError:
        return None
    ent = table.get(traffic_key(kernel, workload, precision))
    if not ent or ent.get("kernels_sha") != kernel_source_digest(kernel, precision):
        return None
    return ent.get("bytes_per_launch")


# Source file that defines each timed kernel, per precision mode (the shared
# headers are hashed with it).
KERNEL_SOURCE = {
    "fp32": {"gemm_fwd": "k_lds.hip", "bwd_fused": "k_lds.hip", "gemm_bwd": "k_gemm.hip",
             "m3_fwd": "k_m3.hip", "m3_bwd": "k_m3.hip", "ce": "k_misc.hip",
             "pack_x": "k_misc.hip", "aux": "k_misc.hip"},
    "bf16": {"gemm_fwd": "k_gemm_bf16.hip", "gemm_bwd": "k_gemm_bf16.hip",
             "m3_fwd": "k_m3.hip", "m3_bwd": "k_m3.hip", "ce": "k_misc.hip",
             "pack_x": "k_misc.hip", "aux": "k_misc.hip"},
}


def kernel_source_digest(kernel: str = None, precision: str = "fp32") -> str:
    """sha256 (16 hex digits) over the source of one kernel and the shared
    headers (all HIP sources when the kernel is not named)."""
    csrc = os.path.join(ROOT, "paper_2206_08369_amd", "csrc")
    names = sorted(n for n in os.listdir(csrc) if n.endswith((".hip", ".h")))
    src = KERNEL_SOURCE.get(precision, {}).get(kernel) if kernel else None
    if src:
        names = sorted(n for n in names if n.endswith(".h") or n == src)
    h = hashlib.sha256()
    for name in names:
        h.update(name.encode())
        h.update(open(os.path.join(csrc, name), "rb").read())
    return h.hexdigest()[:16]


def cpu_baseline(w, hs, acts, X, y, seconds_hint: float):
    """Oracle (every MLP trained alone, fp64, OpenMP over models) on a bounded
    sample of the same workload: all models (or every k-th one when a single
    batch of the whole pack would exceed the time budget) for as many batches
    as fit in about `seconds_hint` seconds.  The oracle's cost is linear in
    each model's width, so a strided sample is scaled by total hidden units."""
    import oracle
    oracle.build(force=False)
    cores = len(os.sched_getaffinity(0))
    if os.environ.get("OMP_NUM_THREADS", "").isdigit():
        cores = max(1, min(cores, int(os.environ["OMP_NUM_THREADS"])))
    N = int(hs.sum())
    flop_batch = (4.0 * w.F + 6.0 * w.O) * N * w.B      # forward + backward + update
    est_rate = 3.5e9 * cores                              # measured order for the plain loops
    est_batch = flop_batch / est_rate
    if est_batch <= seconds_hint:
        stride, nb = 1, int(max(1, min(w.S // w.B, seconds_hint // est_batch)))
    else:
        stride, nb = int(np.ceil(est_batch / seconds_hint)), 1
    models = np.arange(0, w.M, stride)
    W1, W2 = oracle.init_params(w.F, w.O, hs[models], 1)   # any weights: cost is data-independent
    batches = [(k * w.B, w.B) for k in range(nb)]
    t0 = time.perf_counter()
    oracle.train(hs[models], acts[models], W1, W2, X, y, batches, w.lr, nthreads=cores)
    dt = time.perf_counter() - t0
    sub_h = float(hs[models].sum())
    rate = w.M * w.B * nb / (dt * N / sub_h)
    what = ("all %d models" % w.M if stride == 1 else
            "every %d-th model (%d of %d models, %d of %d hidden units)"
            % (stride, len(models), w.M, int(sub_h), N))
    return {
        "value": rate, "unit": "model-samples/s", "cores": oracle.max_threads(),
        "kind": "oracle",
        "sample": "%s, %d batch(es) of %d samples, fp64, %.1f s%s"
                  % (what, nb, w.B, dt, "" if stride == 1 else
                     "; rate scaled to the full pack by total hidden units"),
    }


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=40)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="w10k_f100", choices=sorted(wl.WORKLOADS))
    ap.add_argument("--precision", default="fp32", choices=["fp32", "bf16"])
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="approximate CPU time of the oracle baseline sample (0 = skip)")
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="before timing, run a plain device copy of this many MiB (a known-size "
                         "reference dispatch for hardware byte counters)")
    args = ap.parse_args(argv)

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the packed models are independent, so "
              "a multi-GPU run would shard the model list with no per-step exchange; "
              "that path is not built here.", file=sys.stderr)
        return 2

    import torch
    import paper_2206_08369_amd as pm

    torch.cuda.set_device(0)
    w = wl.WORKLOADS[args.workload]
    hs, acts = w.model_grid()
    X, y = wl.workload_dataset(w)
    N, M = int(hs.sum()), w.M
    Xd = torch.from_numpy(X).cuda()
    yd = torch.from_numpy(y).cuda()
    nfull = w.S // w.B
    net = pm.PackedMLP(w.F, w.O, hs, acts, seed=w.init_seed,
                       precision=pm.PMLP_BF16_GEMM if args.precision == "bf16" else pm.PMLP_FP32)

    def step(k):
        s = (k % nfull) * w.B
        net.train_step(Xd[s:s + w.B], yd[s:s + w.B], w.lr)

    if args.copy_probe_mib > 0:
        n = args.copy_probe_mib * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(2):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    for k in range(args.warmup):
        step(k)
    torch.cuda.synchronize()
    net.profile_reset()
    net.set_profiling(True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(args.steps):
        step(args.warmup + k)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    times = net.kernel_times()
    net.set_profiling(False)
    losses = net.losses()
    if not np.all(np.isfinite(losses)):
        print("non-finite losses after the timed steps", file=sys.stderr)
        return 1

    ms_per_step = 1e3 * elapsed / args.steps
    value = M * w.B * args.steps / elapsed
    kernels = {}
    for name, (ms, n) in times.items():
        if n == 0:
            continue
        bound, nbytes, flops = kernel_work(name, w.B, w.F, N, M, w.O, args.precision)
        avg = ms / n
        kernels[name] = {"avg_ms": avg, "launches": n,
                         "gbs": nbytes / (avg * 1e-3) / 1e9 if nbytes else None,
                         "tflops": flops / (avg * 1e-3) / 1e12 if flops else None}
    dom = max(kernels, key=lambda k: kernels[k]["avg_ms"] * kernels[k]["launches"])
    bound, nbytes, flops = kernel_work(dom, w.B, w.F, N, M, w.O, args.precision)
    mpeak = mfma_peak(dom, w.B, w.F, w.O, args.precision)
    bound = roofline_bound(bound, nbytes, flops, mpeak)
    avg_s = kernels[dom]["avg_ms"] * 1e-3
    if bound == "mfma":
        peak = mpeak
        achieved, unit = flops / avg_s / 1e12, "TFLOP/s"
    else:
        peak, achieved, unit = PEAK_HBM_GBS, nbytes / avg_s / 1e9, "GB/s"
    roofline = {"bound": bound, "achieved": achieved, "peak": peak, "unit": unit,
                "frac": achieved / peak, "traffic": load_traffic(dom, w.name, args.precision),
                "kernel": dom,
                # the kernel's matrix-core ceiling in TFLOP/s of fp32 work, which sets
                # the ridge that chose `bound` (a sixth of the bf16 peak where the
                # products run as six bf16 products of three-piece splits)
                "mfma_ceiling": mpeak,
                "three_piece": args.precision == "fp32" and three_piece(dom, w.B, w.F, w.O)}

    cpu = None
    if args.cpu_seconds > 0:
        cpu = cpu_baseline(w, hs, acts, X, y, args.cpu_seconds)

    line = {
        "metric": METRIC, "value": value, "unit": "model-samples/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms_per_step,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f32" if args.precision == "fp32" else "bf16-gemm/f32",
        "data": "synthetic (seeded X ~ N(0,1), linear-teacher labels; seeded weight init)",
        "config": {"workload": w.name, "models": M, "hidden_units": N, "F": w.F, "O": w.O,
                   "batch": w.B, "samples": w.S, "hidden_sizes": "%d..%d" % w.sizes,
                   "activations": len(w.acts)},
        "roofline": roofline,
        "cpu_baseline": cpu,
        "kernels": kernels,
    }
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
