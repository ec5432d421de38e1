"""Benchmark: packed ParallelMLPs SGD training on one MI355X.

One step = one batch through the whole hot path (batch packing, the
input-layer product, activation + M3 forward, per-model softmax
cross-entropy, the fused backward with both SGD updates).  Steps run in
epoch order: contiguous batches of the workload's samples, the last partial
batch included (Section 4.3 trains whole epochs), starting at an epoch
boundary.  Inputs are seeded synthetic data shaped like the paper's
simulated workloads, resident in GPU memory before timing; weights start
from the library's seeded initialisation.

Prints ONE JSON line: whole-window throughput in model-samples trained per
second, the median over the whole epochs inside the timed window, the
roofline position of the dominant kernel (per-kernel times from HIP events
on the library's stream, taken in a separate profiled epoch so the timed
window runs without them) and the CPU oracle's rate on a bounded sample of
the same workload.  With --graph each epoch is captured once as a HIP graph
and replayed (for packs small enough that launch overhead matters).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
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
    flops count multiply-adds as two operations.  The bf16 storage mode also
    keeps Z in bf16 (2 bytes per element wherever Z is written or read)."""
    f4 = 4.0
    bf = precision in ("bf16", "bf16_store")
    fx = 2.0 if bf else 4.0      # bytes per element of the batch copy
    fz = 2.0 if precision == "bf16_store" else 4.0   # bytes per element of Z
    if name == "gemm_fwd":       # Z = X W1^T: read W1 (bf16 copy in bf16 mode), X; write Z
        return "mfma", (2.0 if bf else f4) * N * F + fx * B * F + fz * N * B, 2.0 * B * F * N
    if name == "gemm_bwd":       # W1 -= lr dZ^T X: read dZ, X; read+write W1 (+ its bf16 copy)
        return ("mfma", (2.0 if bf else f4) * N * B + fx * B * F + 2 * f4 * N * F
                + (2.0 * N * F if bf else 0.0), 2.0 * B * F * N)
    if name == "fwd_m3":         # one kernel: read W1, X, W2; write Z and the logits
        return ("mfma", f4 * (N * F + B * F + N * B + O * N + B * M * O),
                2.0 * B * F * N + 2.0 * B * O * N)
    if name == "m3_fwd":         # read Z, W2; write logits
        return "hbm", fz * N * B + f4 * (O * N + B * M * O), 2.0 * B * O * N
    if name == "m3_bwd":         # read Z, G, W2; write dZ (bf16 in bf16 mode), W2
        return ("hbm", fz * N * B + (2.0 if bf else f4) * N * B + f4 * (2 * O * N + B * M * O),
                4.0 * B * O * N)
    if name == "bwd_fused":      # read Z, G, X; read+write W1 and W2 (dZ stays in registers)
        return ("mfma", f4 * (N * B + B * M * O + B * F + 2 * N * F + 2 * O * N),
                2.0 * B * F * N + 4.0 * B * O * N)
    if name == "ce":             # read logits, y; write G, loss
        return "hbm", f4 * (2 * B * M * O + B + M), 0.0
    if name == "pack_x":         # read X; write two padded copies
        return "hbm", f4 * B * F + 2 * fx * B * F, 0.0
    return "hbm", 0.0, 0.0


# Matrix-core ceiling of a kernel, by the arithmetic the library reports it
# ran (PMLP_ARITH_*), in TFLOP/s of the kernel's own (fp32-equivalent) work.
ARITH_CEILING = {
    1: PEAK_FP32_MFMA,            # fp32 matrix cores
    2: PEAK_BF16_MFMA / 6.0,      # six bf16 products of three-piece splits per fp32 product
    3: PEAK_BF16_MFMA,            # bf16 operands, fp32 accumulation
}


def mfma_peak(arith: int):
    """Matrix-core ceiling for a PMLP_ARITH_* code, or None (no matrix work)."""
    return ARITH_CEILING.get(arith)


def roofline_bound(bound, nbytes, flops, peak_tflops):
    """A matrix-core kernel is compute-bound only when its arithmetic
    intensity (algorithmic flops per algorithmic byte) is above the ridge
    point of its matrix-core ceiling (peak flops / peak HBM bandwidth);
    below it the HBM roofline bounds it."""
    if bound != "mfma" or not nbytes or not peak_tflops:
        return "hbm" if bound == "mfma" else bound
    ridge = peak_tflops * 1e12 / (PEAK_HBM_GBS * 1e9)
    return "mfma" if flops / nbytes >= ridge else "hbm"


def traffic_key(kernel: str, workload: str, precision: str) -> str:
    return "%s/%s%s" % (kernel, workload, "" if precision == "fp32" else "+" + precision)


def load_traffic(kernel: str, workload: str, precision: str = "fp32"):
    """HBM bytes per launch from committed rocprofv3 counter summaries, if
    they were taken on the current source of the kernel they name; otherwise
    None."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    try:
        table = json.load(open(path))
    except ValueError:
        return None
    ent = table.get(traffic_key(kernel, workload, precision))
    if not ent or ent.get("kernels_sha") != kernel_source_digest(ent.get("kernel", "")):
        return None
    return ent.get("bytes_per_launch")


# variants the library reports under their own name that are instances of
# another kernel
VARIANT_KERNEL = {"k_gemm_x3": "k_gemm_bf"}


def kernel_source(kernel: str):
    """Source file (under csrc/) that defines a kernel, given the name the
    library reports or a trace shows (template arguments are ignored)."""
    base = kernel.split("<")[0].strip()
    base = VARIANT_KERNEL.get(base, base)
    csrc = os.path.join(ROOT, "paper_2206_08369_amd", "csrc")
    pat = re.compile(r"\bvoid\s+%s\s*\(" % re.escape(base))
    for name in sorted(os.listdir(csrc)):
        if name.endswith(".hip") and pat.search(open(os.path.join(csrc, name)).read()):
            return name
    return None


def kernel_source_digest(kernel: str = None) -> str:
    """sha256 (16 hex digits) over the source file of one kernel and the
    shared headers (all HIP sources when the kernel is not named or not
    found)."""
    csrc = os.path.join(ROOT, "paper_2206_08369_amd", "csrc")
    names = sorted(n for n in os.listdir(csrc) if n.endswith((".hip", ".h")))
    src = kernel_source(kernel) if kernel else None
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


def measured_hbm(torch, gib: int = 2):
    """GB/s of plain device streams: a sum (read), a fill (write) and a copy
    (read + write, counted both ways) over `gib` GiB, best of three each."""
    n = gib * (1 << 30) // 4
    a = torch.ones(n, dtype=torch.float32, device="cuda")
    b = torch.empty_like(a)
    out = {}
    for name, fn, nbytes in (("read", lambda: a.sum(), 4 * n), ("write", lambda: b.fill_(2.0), 4 * n),
                             ("copy", lambda: b.copy_(a), 8 * n)):
        best = None
        for _ in range(4):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            fn()
            e1.record()
            torch.cuda.synchronize()
            ms = e0.elapsed_time(e1)
            best = ms if best is None else min(best, ms)
        out[name] = nbytes / (best * 1e-3) / 1e9
    del a, b
    torch.cuda.empty_cache()
    out["unit"] = "GB/s"
    out["how"] = "torch sum / fill_ / copy_ over %d GiB fp32, best of 3 after one warm-up" % gib
    return out


def epoch_batches(w):
    """(offset, length) of every batch of one epoch, the partial one last."""
    return w.batches()


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None,
                    help="timed steps, in epoch order from an epoch boundary "
                         "(default: three whole epochs)")
    ap.add_argument("--warmup", type=int, default=None,
                    help="untimed steps before (default: one whole epoch)")
    ap.add_argument("--workload", default="w10k_f100", choices=sorted(wl.WORKLOADS))
    ap.add_argument("--precision", default="fp32", choices=["fp32", "bf16", "bf16_store"],
                    help="bf16: the bf16 operand mode (PMLP_BF16_GEMM); bf16_store: with Z "
                         "also stored in bf16 (PMLP_BF16_STORE)")
    ap.add_argument("--graph", action="store_true",
                    help="capture one epoch as a HIP graph and replay it (timed steps are "
                         "rounded up to whole epochs)")
    ap.add_argument("--no-partial", action="store_true",
                    help="leave each epoch's partial last batch out (profiling runs, so that "
                         "per-kernel averages are those of full-batch launches)")
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
    batches = epoch_batches(w)
    if args.no_partial:
        batches = [b for b in batches if b[1] == w.B]
    spe = len(batches)
    steps = args.steps if args.steps is not None else 3 * spe
    warmup = args.warmup if args.warmup is not None else spe
    if args.graph:
        steps = spe * max(1, -(-steps // spe))
    mode = {"fp32": pm.PMLP_FP32, "bf16": pm.PMLP_BF16_GEMM,
            "bf16_store": pm.PMLP_BF16_STORE}[args.precision]
    net = pm.PackedMLP(w.F, w.O, hs, acts, seed=w.init_seed, precision=mode)

    def step(k):
        s, n = batches[k % spe]
        net.train_step(Xd[s:s + n], yd[s:s + n], w.lr)

    if args.copy_probe_mib > 0:
        n = args.copy_probe_mib * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(2):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    # warm-up ends on an epoch boundary so the timed window starts one
    warm = -(-warmup // spe) * spe if warmup else 0
    for k in range(warm):
        step(k)
    graph = None
    if args.graph:
        graph = torch.cuda.CUDAGraph()
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            step(0)                   # one eager step on the capture stream
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        with torch.cuda.graph(graph, capture_error_mode="relaxed"):
            for k in range(spe):
                step(k)
        torch.cuda.synchronize()
    samples = [batches[k % spe][1] for k in range(steps)]
    marks = []
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    start = torch.cuda.Event(enable_timing=True)
    start.record()
    if graph is not None:
        for _ in range(steps // spe):
            graph.replay()
            ev = torch.cuda.Event(enable_timing=True)
            ev.record()
            marks.append(ev)
    else:
        for k in range(steps):
            step(k)
            if (k + 1) % spe == 0:
                ev = torch.cuda.Event(enable_timing=True)
                ev.record()
                marks.append(ev)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    losses = net.losses()
    if not np.all(np.isfinite(losses)):
        print("non-finite losses after the timed steps", file=sys.stderr)
        return 1
    epoch_s = []
    prev = start
    for ev in marks:
        epoch_s.append(prev.elapsed_time(ev) * 1e-3)
        prev = ev

    # per-kernel times: the full batches of one more epoch, with HIP events
    # around every launch (the roofline figures are per full-batch launch)
    net.profile_reset()
    net.set_profiling(True)
    for k in range(spe):
        if batches[k][1] == w.B:
            step(k)
    torch.cuda.synchronize()
    times = net.kernel_times()
    variants = net.kernel_variants()
    net.set_profiling(False)

    value = M * float(sum(samples)) / elapsed
    ms_per_step = 1e3 * elapsed / steps
    kernels = {}
    for name, (ms, n) in times.items():
        if n == 0:
            continue
        bound, nbytes, flops = kernel_work(name, w.B, w.F, N, M, w.O, args.precision)
        avg = ms / n
        kernels[name] = {"avg_ms": avg, "launches": n, "kernel": variants[name][0],
                         "gbs": nbytes / (avg * 1e-3) / 1e9 if nbytes else None,
                         "tflops": flops / (avg * 1e-3) / 1e12 if flops else None}
    dom = max(kernels, key=lambda k: kernels[k]["avg_ms"] * kernels[k]["launches"])
    bound, nbytes, flops = kernel_work(dom, w.B, w.F, N, M, w.O, args.precision)
    arith = variants[dom][1]
    mpeak = mfma_peak(arith)
    bound = roofline_bound(bound, nbytes, flops, mpeak)
    avg_s = kernels[dom]["avg_ms"] * 1e-3
    if bound == "mfma":
        peak = mpeak
        achieved, unit = flops / avg_s / 1e12, "TFLOP/s"
    else:
        peak, achieved, unit = PEAK_HBM_GBS, nbytes / avg_s / 1e9, "GB/s"
    roofline = {"bound": bound, "achieved": achieved, "peak": peak, "unit": unit,
                "frac": achieved / peak, "traffic": load_traffic(dom, w.name, args.precision),
                "kernel": dom, "kernel_name": variants[dom][0],
                # the matrix-core ceiling (TFLOP/s of the kernel's fp32-equivalent work)
                # of the arithmetic the library reports the kernel ran; it sets the
                # ridge that chose `bound`
                "mfma_ceiling": mpeak, "arith": arith}

    # what this GPU's HBM sustains for plain streams (torch reductions, fills
    # and copies over 2 GiB, best of three): the practical ceiling the
    # memory-bound kernels are read against, beside the published peak
    hbm = measured_hbm(torch)
    roofline["frac_of_measured_copy"] = (achieved / hbm["copy"] if unit == "GB/s" else None)
    nfull = sum(1 for _, n in batches if n == w.B)
    step_bytes = 0.0
    for name, (ms, n) in times.items():
        if n:
            step_bytes += kernel_work(name, w.B, w.F, N, M, w.O, args.precision)[1] * n / nfull

    cpu = None
    if args.cpu_seconds > 0:
        cpu = cpu_baseline(w, hs, acts, X, y, args.cpu_seconds)

    med = float(np.median(epoch_s)) if epoch_s else None
    line = {
        "metric": METRIC, "value": value, "unit": "model-samples/s", "n_gpus": 1,
        "steps": steps, "warmup": warm, "ms_per_step": ms_per_step,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": {"fp32": "f32", "bf16": "bf16-gemm/f32",
                  "bf16_store": "bf16-gemm/bf16-z/f32"}[args.precision],
        "data": "synthetic (seeded X ~ N(0,1), linear-teacher labels; seeded weight init)",
        "config": {"workload": w.name, "models": M, "hidden_units": N, "F": w.F, "O": w.O,
                   "batch": w.B, "samples": w.S, "hidden_sizes": "%d..%d" % w.sizes,
                   "activations": len(w.acts), "steps_per_epoch": spe, "graph": bool(graph),
                   "partial_batches": not args.no_partial},
        "epochs": {"count": len(epoch_s), "median_s": med,
                   "value_median": M * sum(n for _, n in batches) / med if med else None,
                   "all_s": epoch_s},
        "roofline": roofline,
        "hbm_measured": hbm,
        # algorithmic HBM bytes of one full-batch step (all kernels) and the
        # rate they move at over the timed steps
        "step_traffic": {"bytes": step_bytes, "gbs": step_bytes / (ms_per_step * 1e-3) / 1e9},
        "cpu_baseline": cpu,
        "kernels": kernels,
    }
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
