"""Summaries of rocprofv3 runs of bench.py for profiles/ (run on the host
after the runs; reads their CSV output, writes Markdown tables and the
per-kernel HBM traffic table that bench.py reports).

The runs (one MI355X; from /tmp with TMPDIR=/tmp; $R = repository root,
$W = workload, $P = precision, $O = an output directory):

  trace:  rocprofv3 --kernel-trace --stats -f csv -d $O/trace -o run -- \\
              python3 $R/bench.py --workload $W --precision $P --steps 3 --warmup 1 \\
              --cpu-seconds 0 --no-partial
  set A:  rocprofv3 --pmc SQ_WAVES SQ_BUSY_CYCLES SQ_WAVE_CYCLES SQ_WAIT_INST_ANY \\
              SQ_ACTIVE_INST_VALU SQ_ACTIVE_INST_LDS SQ_VALU_MFMA_BUSY_CYCLES \\
              SQ_LDS_BANK_CONFLICT GRBM_GUI_ACTIVE --kernel-trace -f csv -d $O/A -o run -- \\
              python3 $R/bench.py (same arguments)
  set B:  rocprofv3 --pmc SQ_INSTS_VALU SQ_INSTS_LDS SQ_INSTS_SALU SQ_INSTS_VMEM_RD \\
              SQ_INSTS_VMEM_WR SQ_ACTIVE_INST_VMEM SQ_ACTIVE_INST_ANY SQ_WAIT_ANY \\
              GRBM_GUI_ACTIVE --kernel-trace -f csv -d $O/B -o run -- python3 $R/bench.py ...
  fetch:  rocprofv3 --pmc FETCH_SIZE --kernel-trace -f csv -d $O/FETCH_SIZE -o run -- \\
              python3 $R/bench.py ... --copy-probe-mib 1024
  write:  the same with WRITE_SIZE

  set C:  rocprofv3 --pmc SQ_VALU_MFMA_COEXEC_CYCLES SQ_VALU_MFMA_BUSY_CYCLES SQ_INSTS_MFMA \\
              SQ_INSTS_VALU_TRANS_F32 GRBM_GUI_ACTIVE --kernel-trace -f csv -d $O/C -o run -- \\
              python3 $R/bench.py ...   (optional)

and the benchmark's own line, `python3 $R/bench.py ... > $O/bench.json`.  With
--label L and --env NAME=VALUE the runs were made with that environment
setting (for instance PMLP_FUSED_FORWARD=1) and the files are named for
WORKLOAD_L.

usage: python bench_profiles.py OUTDIR WORKLOAD [PRECISION] [--label L --env NAME=VALUE]
"""
from __future__ import annotations

import collections
import csv
import glob
import json
import os
import re
import sys

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import bench  # noqa: E402

def agent(outdir: str):
    """(SIMDs, XCDs) of the GPU the counters were taken on (rocprofv3's agent table)."""
    for r in rows(os.path.join(outdir, "A", "**", "*agent_info.csv")):
        if r.get("Name", "").startswith("gfx"):
            return int(r["Simd_Count"]), int(r["Num_Xcc"])
    return 1024, 8   # MI355X: 256 CUs x 4 SIMDs, 8 XCDs

# kernel (template base name) -> bench.py role
ROLE = {
    "k_pack_x": "pack_x", "k_pack_x_bf16": "pack_x", "k_fwd_lds": "gemm_fwd",
    "k_fwd_lds_ring": "gemm_fwd", "k_fwd_x3": "gemm_fwd", "k_fwd_x3m": "fwd_m3",
    "k_m3_fwd": "m3_fwd",
    "k_m3_fwd_mf": "m3_fwd", "k_ce": "ce", "k_mse": "ce", "k_fill": "aux",
    "k_bwd_lds": "bwd_fused", "k_bwd_x3": "bwd_fused", "k_bwd_mf": "bwd_fused",
    "k_m3_bwd": "m3_bwd", "k_w1_to_bf16": "aux",
}

SET_A = ("SQ_WAVES SQ_BUSY_CYCLES SQ_WAVE_CYCLES SQ_WAIT_INST_ANY SQ_ACTIVE_INST_VALU "
         "SQ_ACTIVE_INST_LDS SQ_VALU_MFMA_BUSY_CYCLES SQ_LDS_BANK_CONFLICT GRBM_GUI_ACTIVE")
SET_B = ("SQ_INSTS_VALU SQ_INSTS_LDS SQ_INSTS_SALU SQ_INSTS_VMEM_RD SQ_INSTS_VMEM_WR "
         "SQ_ACTIVE_INST_VMEM SQ_ACTIVE_INST_ANY SQ_WAIT_ANY GRBM_GUI_ACTIVE")
SET_C = ("SQ_VALU_MFMA_COEXEC_CYCLES SQ_VALU_MFMA_BUSY_CYCLES SQ_INSTS_MFMA SQ_INSTS_VALU_TRANS_F32 "
         "GRBM_GUI_ACTIVE")


def short(name: str) -> str:
    n = name.replace("(anonymous namespace)::", "").replace("pmlpk::", "").replace("void ", "")
    return re.sub(r"\(.*", "", n).strip()


def role_of(name: str, precision: str):
    base = name.split("<")[0]
    if base == "k_gemm_bf" or base == "k_gemm_nt":
        # the epilogue: last argument of k_gemm_nt, the one after the operand
        # type flag of k_gemm_bf
        args = [a.strip() for a in name.split("<", 1)[-1].rstrip(">").split(",")]
        if base == "k_gemm_bf":
            flags = [i for i, a in enumerate(args) if a in ("true", "false")]
            epi = args[flags[0] + 1] if flags and flags[0] + 1 < len(args) else ""
        else:
            epi = args[-1]
        return {"0": "gemm_fwd", "1": "gemm_bwd", "2": "gemm_grad"}.get(epi, "gemm")
    return ROLE.get(base)


def rows(path_glob: str):
    out = []
    for p in sorted(glob.glob(path_glob, recursive=True)):
        with open(p, newline="") as f:
            out.extend(csv.DictReader(f))
    return out


def kernel_trace(outdir: str):
    """{kernel: [durations in us]} from the kernel-trace CSV."""
    per = collections.defaultdict(list)
    for r in rows(os.path.join(outdir, "trace", "**", "*kernel_trace.csv")):
        name = short(r["Kernel_Name"])
        per[name].append((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-3)
    return per


def counters(outdir: str, tag: str):
    """{kernel: {counter: [value per dispatch]}}."""
    per = collections.defaultdict(lambda: collections.defaultdict(list))
    disp = collections.defaultdict(dict)
    for r in rows(os.path.join(outdir, tag, "**", "*counter_collection.csv")):
        name = short(r["Kernel_Name"])
        did = r.get("Dispatch_Id") or r.get("Correlation_Id")
        disp[(name, did)][r["Counter_Name"]] = float(r["Counter_Value"])
    for (name, _), cs in disp.items():
        for c, v in cs.items():
            per[name][c].append(v)
    return per


def mean(v):
    return sum(v) / len(v) if v else float("nan")


def main(argv):
    if len(argv) < 2:
        print(__doc__)
        return 2
    label, env = None, None
    pos = []
    it = iter(argv)
    for a in it:
        if a == "--label":
            label = next(it)
        elif a == "--env":
            env = next(it)
        else:
            pos.append(a)
    outdir, wk = pos[0], pos[1]
    prec = pos[2] if len(pos) > 2 else "fp32"
    tag = wk if prec == "fp32" else "%s_%s" % (wk, prec)
    if label:
        tag += "_" + label
    envp = (env + " ") if env else ""
    b = json.load(open(os.path.join(outdir, "bench.json")))
    cfg = b["config"]
    N, M, F, O, B = cfg["hidden_units"], cfg["models"], cfg["F"], cfg["O"], cfg["batch"]
    args = "--workload %s%s --steps 3 --warmup 1 --cpu-seconds 0 --no-partial" % (
        wk, "" if prec == "fp32" else " --precision " + prec)
    head = "# %%s: `%s` (%d models, N = %s, F = %d, O = %d, B = %d), %s%s\n" % (
        wk, M, format(N, ","), F, O, B, prec, (", with " + env) if env else "")

    # kernel trace
    tr = kernel_trace(outdir)
    lines = [head % "Kernel trace", "Command (one MI355X, from /tmp with TMPDIR=/tmp; $R = repository root):", "",
             "```", envp + "rocprofv3 --kernel-trace --stats -f csv -d $R/gpurun_out/prof/%s/trace -o run -- \\" % tag,
             "    python3 $R/bench.py %s" % args, "python3 $R/bench_profiles.py $R/gpurun_out/prof/%s %s %s%s"
             % (tag, wk, prec, (" --label %s --env %s" % (label, env)) if label else ""), "```", "",
             "Every launch of the run (warm-up epoch, timed steps and the profiled epoch, full batches only):", "",
             "| kernel (role) | calls | avg (us) | min (us) | max (us) | % of GPU time |",
             "|---|---:|---:|---:|---:|---:|"]
    total = sum(sum(v) for v in tr.values())
    for name, d in sorted(tr.items(), key=lambda kv: -sum(kv[1])):
        if name.startswith("__amd"):
            continue
        lines.append("| `%s` (%s) | %d | %.1f | %.1f | %.1f | %.1f |" % (
            name, role_of(name, prec) or "", len(d), mean(d), min(d), max(d),
            100.0 * sum(d) / total))
    lines += ["", "The same kernels timed live by `bench.py` (HIP events on the library stream, "
              "one profiled epoch of full batches, separate run):", "",
              "| role | kernel | avg (us) | achieved |", "|---|---|---:|---|"]
    for k, v in b["kernels"].items():
        a = []
        if v.get("tflops"):
            a.append("%.1f TFLOP/s" % v["tflops"])
        if v.get("gbs"):
            a.append("%.0f GB/s" % v["gbs"])
        lines.append("| %s | `%s` | %.1f | %s |" % (k, v.get("kernel", ""), v["avg_ms"] * 1e3,
                                                   ", ".join(a)))
    lines += ["", "Timed window of that run: %.3f ms/step, %.4g model-samples/s." % (
        b["ms_per_step"], b["value"])]
    open(os.path.join(ROOT, "profiles", "kernel_trace_%s.md" % tag), "w").write("\n".join(lines) + "\n")

    # counters (only where the counter passes were taken)
    ca, cb = counters(outdir, "A"), counters(outdir, "B")
    if not ca:
        return 0
    simds, nxcc = agent(outdir)
    lines = [head % "Counters", "Two counter passes, each in its own run (arguments of bench.py as in "
             "`kernel_trace_%s.md`):" % tag, "", "```",
             envp + "rocprofv3 --pmc %s --kernel-trace -f csv -d $R/gpurun_out/prof/%s/A -o run -- python3 $R/bench.py %s"
             % (SET_A, tag, args),
             envp + "rocprofv3 --pmc %s --kernel-trace -f csv -d $R/gpurun_out/prof/%s/B -o run -- python3 $R/bench.py %s"
             % (SET_B, tag, args),
             envp + "rocprofv3 --pmc %s --kernel-trace -f csv -d $R/gpurun_out/prof/%s/C -o run -- python3 $R/bench.py %s"
             % (SET_C, tag, args), "```", "",
             "Per kernel, means over its dispatches.  GRBM_GUI_ACTIVE is summed over the %d XCDs, "
             "so T = GRBM_GUI_ACTIVE / %d is the kernel's active cycles.  Derived columns:" % (nxcc, nxcc), "",
             "- MFMA busy = SQ_VALU_MFMA_BUSY_CYCLES / (T x %d SIMDs)" % simds,
             "- VALU busy = 4 x SQ_ACTIVE_INST_VALU / (T x %d SIMDs) (rocprof's VALUBusy)" % simds,
             "- issue wait = SQ_WAIT_INST_ANY / SQ_WAVE_CYCLES (share of wave time with an instruction "
             "ready but not issued)",
             "- s_waitcnt = SQ_WAIT_ANY / SQ_WAVE_CYCLES (share of wave time in s_waitcnt, pass B)",
             "- LDS conflicts = SQ_LDS_BANK_CONFLICT / SQ_ACTIVE_INST_LDS",
             "- clock = T / kernel duration (duration from the trace of the same run)",
             "- co-exec = SQ_VALU_MFMA_COEXEC_CYCLES / (T x %d SIMDs): cycles in which a vector "
             "instruction issued while the matrix pipe was busy (pass C, where taken)" % simds, "",
             "| kernel | MFMA busy | VALU busy | co-exec | issue wait | s_waitcnt | LDS conflicts | "
             "clock (GHz) | VALU instr / wave | LDS instr / wave | waves |",
             "|---|---:|---:|---:|---:|---:|---:|---:|---:|---:|---:|"]
    cc = counters(outdir, "C")
    nan = float("nan")
    for name in sorted(ca, key=lambda n: -mean(ca[n].get("GRBM_GUI_ACTIVE", [0]))):
        if name.startswith("__amd"):
            continue
        a, bb, c3 = ca[name], cb.get(name, {}), cc.get(name, {})
        g = mean(a["GRBM_GUI_ACTIVE"]) / nxcc
        d = mean(tr.get(name, [])) if tr.get(name) else nan
        waves = mean(a["SQ_WAVES"])
        co = (mean(c3["SQ_VALU_MFMA_COEXEC_CYCLES"]) / ((mean(c3["GRBM_GUI_ACTIVE"]) / nxcc) * simds)
              if c3 else nan)
        lines.append("| `%s` | %.2f | %.2f | %.2f | %.2f | %.2f | %.3f | %.2f | %.0f | %.0f | %.0f |" % (
            name, mean(a["SQ_VALU_MFMA_BUSY_CYCLES"]) / (g * simds),
            4 * mean(a["SQ_ACTIVE_INST_VALU"]) / (g * simds), co,
            mean(a["SQ_WAIT_INST_ANY"]) / max(mean(a["SQ_WAVE_CYCLES"]), 1.0),
            mean(bb.get("SQ_WAIT_ANY", [nan])) / max(mean(a["SQ_WAVE_CYCLES"]), 1.0),
            mean(a["SQ_LDS_BANK_CONFLICT"]) / max(mean(a["SQ_ACTIVE_INST_LDS"]), 1.0),
            g / (d * 1e3) if d == d else nan,
            mean(bb.get("SQ_INSTS_VALU", [nan])) / max(waves, 1.0),
            mean(bb.get("SQ_INSTS_LDS", [nan])) / max(waves, 1.0), waves))
    open(os.path.join(ROOT, "profiles", "counters_%s.md" % tag), "w").write("\n".join(lines) + "\n")

    # traffic, calibrated on plain kernels of known size in the same runs:
    # bench.py's HBM probe sums 2 GiB (a read-only reduction) and fills
    # 2 GiB (a write-only elementwise kernel); HIP's device copy is listed too
    fs = counters(outdir, "FETCH_SIZE")
    ws = counters(outdir, "WRITE_SIZE")
    if not fs or not ws:
        return 0
    kib = 1024.0 * 1024.0
    ref = 2.0 * kib   # KiB each probe kernel moves
    red = [n for n in fs if "reduce_kernel" in n and "sum_functor" in n]
    fil = [n for n in ws if "FillFunctor" in n]
    cf = ref / max(fs[red[0]]["FETCH_SIZE"])
    cw = ref / max(ws[fil[0]]["WRITE_SIZE"])
    copy = [n for n in fs if n.startswith("__amd_rocclr_copyBuffer")]
    copy_note = ""
    if copy and copy[0] in ws:
        copy_note = (" For comparison, HIP's device-to-device copy of 1 GiB (`--copy-probe-mib 1024`) "
                     "reads FETCH_SIZE = %.0f KiB and WRITE_SIZE = %.0f KiB for 1,048,576 KiB each "
                     "way; its counts differ from one box to another and from how the counters read "
                     "the kernels here, so it is not the reference." % (
                         max(fs[copy[0]]["FETCH_SIZE"]), max(ws[copy[0]]["WRITE_SIZE"])))
    tpath = os.path.join(ROOT, "profiles", "traffic.json")
    table = json.load(open(tpath)) if os.path.exists(tpath) else {}
    lines = [head % "HBM traffic per launch", "Two counter passes (KiB per dispatch), each in its own run:", "",
             "```", envp + "rocprofv3 --pmc FETCH_SIZE --kernel-trace -f csv -d $R/gpurun_out/prof/%s/FETCH_SIZE -o run -- "
             "python3 $R/bench.py %s --copy-probe-mib 1024" % (tag, args),
             envp + "rocprofv3 --pmc WRITE_SIZE --kernel-trace -f csv -d $R/gpurun_out/prof/%s/WRITE_SIZE -o run -- "
             "python3 $R/bench.py %s --copy-probe-mib 1024" % (tag, args), "```", "",
             "Calibration: in the same runs bench.py sums 2 GiB (torch's reduction, a read-only "
             "stream) and fills 2 GiB (torch's fill, a write-only stream); they read FETCH_SIZE = "
             "%.0f KiB and WRITE_SIZE = %.0f KiB for 2,097,152 KiB moved: scale factors %.3f "
             "(fetch) and %.3f (write).%s" % (ref / cf, ref / cw, cf, cw, copy_note), "",
             "| kernel (role) | FETCH_SIZE (KiB) | WRITE_SIZE (KiB) | HBM bytes (scaled) | algorithmic bytes | ratio |",
             "|---|---:|---:|---:|---:|---:|"]
    for name in fs:
        role = role_of(name, prec)
        if role is None or name not in ws:
            continue
        f_k, w_k = mean(fs[name]["FETCH_SIZE"]), mean(ws[name]["WRITE_SIZE"])
        hbm = 1024.0 * (cf * f_k + cw * w_k)
        _, alg, _ = bench.kernel_work(role, B, F, N, M, O, prec)
        lines.append("| `%s` (%s) | %.0f | %.0f | %.4g | %.4g | %s |" % (
            name, role, f_k, w_k, hbm, alg, "%.3f" % (hbm / alg) if alg else "-"))
        table[bench.traffic_key(role, wk, prec)] = {
            "kernel": name, "bytes_per_launch": hbm, "fetch_kib": f_k, "write_kib": w_k,
            "kernels_sha": bench.kernel_source_digest(name)}
    lines += ["", "Each entry of `profiles/traffic.json` carries the hash of its kernel's source file "
              "and the shared headers; `bench.py` reports `traffic` only while it matches."]
    open(os.path.join(ROOT, "profiles", "traffic_%s.md" % tag), "w").write("\n".join(lines) + "\n")
    json.dump(table, open(tpath, "w"), indent=1, sort_keys=True)
    return 0


if __name__ == "__main__":
    sys.exit(main(sys.argv[1:]))
