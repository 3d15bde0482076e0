"""Summaries under profiles/ from rocprofv3 output.

The passes (each its own rocprofv3 run, counters split so that every pass
fits the counter blocks) are listed in PASSES; `--show-commands DIR` prints
them as shell lines writing under DIR, and `--dir DIR` turns their CSV
output into the committed summaries:

  k_dgrad_rows_ssc128_c64_kernel_stats.txt   kernel trace of the layer step
  k_dgrad_rows_ssc128_c64_traffic.json       FETCH_SIZE / WRITE_SIZE per kernel,
                                             calibrated, with the algorithmic
                                             bytes of the dominant kernel
  ssc128_c64_mfma_counters.txt               MFMA and LDS counters of the
                                             contraction kernels
  rulebook_build_scenes256_traffic.txt       per-kernel time and traffic of the
                                             SSC and SC builds at about 2M sites
  bench_all_workloads_kernel_stats.txt       kernel trace of a whole bench.py run

Calibration: a plain copy of B bytes (the measure library's k_copy) should
read B and write B; FETCH_SIZE and WRITE_SIZE (KiB per dispatch) are scaled
by B / (what they read for that copy).  MFMA busy is
SQ_VALU_MFMA_BUSY_CYCLES / (SIMDs x cycles per XCD), with GRBM_GUI_ACTIVE
summed over the 8 XCDs.  Measurement infrastructure only.
"""
from __future__ import annotations

import argparse
import csv
import glob
import hashlib
import json
import os
import re
from collections import defaultdict

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
PROFILES = os.path.join(ROOT, "profiles")
KERNEL_SRC = os.path.join(ROOT, "paper_1711_10275_amd", "csrc", "conv.hip")
DOMINANT = "k_dgrad_rows<float, 128, 4, 2, 1, false, true>"
N_XCD, N_CU, SIMD_PER_CU = 8, 256, 4

LAYER = "python -u bench.py --steps 3 --warmup 1 --no-extra --no-cpu-baseline --copy-calibration"
BUILDS = "python -u -m paper_1711_10275_amd.measure.builds --reps 3"
PASSES = {
    "trace": ("rocprofv3 --kernel-trace --stats -d {D}/trace -o trace --output-format csv -- "
              "python -u bench.py --steps 10 --warmup 3 --no-extra --no-cpu-baseline", "bench.json"),
    "mfma": ("rocprofv3 --pmc SQ_VALU_MFMA_BUSY_CYCLES SQ_BUSY_CYCLES SQ_INSTS_VALU_MFMA_MOPS_BF16 "
             "SQ_INSTS_VALU_MFMA_MOPS_F32 SQ_INSTS_MFMA SQ_INSTS_VALU SQ_WAVE_CYCLES GRBM_GUI_ACTIVE "
             "-d {D}/mfma -o mfma --output-format csv -- " + LAYER, None),
    "lds": ("rocprofv3 --pmc SQ_ACTIVE_INST_LDS SQ_LDS_BANK_CONFLICT SQ_INSTS_LDS SQ_WAIT_INST_LDS "
            "SQ_ACTIVE_INST_VMEM SQ_WAIT_ANY SQ_BUSY_CYCLES GRBM_GUI_ACTIVE "
            "-d {D}/lds -o lds --output-format csv -- " + LAYER, None),
    "fetch": ("rocprofv3 --pmc FETCH_SIZE -d {D}/fetch -o fetch --output-format csv -- " + LAYER, None),
    "write": ("rocprofv3 --pmc WRITE_SIZE -d {D}/write -o write --output-format csv -- " + LAYER, None),
    "all": ("rocprofv3 --kernel-trace --stats -d {D}/all -o all --output-format csv -- "
            "python -u bench.py --steps 5 --warmup 2 --no-cpu-baseline", "bench_all.json"),
    "btrace": ("rocprofv3 --kernel-trace --stats -d {D}/btrace -o btrace --output-format csv -- " + BUILDS,
               "builds.json"),
    "bfetch": ("rocprofv3 --pmc FETCH_SIZE -d {D}/bfetch -o bfetch --output-format csv -- " + BUILDS, None),
    "bwrite": ("rocprofv3 --pmc WRITE_SIZE -d {D}/bwrite -o bwrite --output-format csv -- " + BUILDS, None),
}


def command(name, d):
    cmd, out = PASSES[name]
    cmd = cmd.format(D=d)
    return cmd + (f" > {d}/{out}" if out else "")


def short(name):
    """Kernel name without return type, namespaces and argument list."""
    s = name.replace("void ", "").replace("(anonymous namespace)::", "").replace("sscn::", "")
    depth, out = 0, []
    for ch in s:  # cut at the argument list's '(' (template arguments have none at depth 0)
        if ch == "(" and depth == 0:
            break
        depth += ch == "<"
        depth -= ch == ">"
        out.append(ch)
    return re.sub(r"\bbf16_t\b", "bf16", "".join(out).strip())


def one_csv(d, suffix):
    files = glob.glob(os.path.join(d, f"*{suffix}"))
    if len(files) != 1:
        raise SystemExit(f"expected one *{suffix} under {d}, found {files}")
    return files[0]


def kernel_stats(d):
    rows = []
    for r in csv.DictReader(open(one_csv(d, "_kernel_stats.csv"))):
        rows.append((short(r["Name"]), int(r["Calls"]), float(r["AverageNs"]) / 1e3, float(r["MinNs"]) / 1e3,
                     float(r["MaxNs"]) / 1e3, float(r["Percentage"])))
    return rows


def counters(d):
    """kernel -> counter -> per-dispatch values (summed over a dispatch's rows)."""
    per = defaultdict(lambda: defaultdict(float))
    names = {}
    for r in csv.DictReader(open(one_csv(d, "_counter_collection.csv"))):
        per[r["Dispatch_Id"]][r["Counter_Name"]] += float(r["Counter_Value"])
        names[r["Dispatch_Id"]] = short(r["Kernel_Name"])
    out = defaultdict(lambda: defaultdict(list))
    for disp, cs in per.items():
        for c, v in cs.items():
            out[names[disp]][c].append(v)
    return out


def mean(xs):
    return sum(xs) / len(xs)


def calibrated_traffic(fetch_dir, write_dir, copy_bytes=256 << 20):
    fe, wr = counters(fetch_dir), counters(write_dir)
    fk, wk = mean(fe["k_copy"]["FETCH_SIZE"]), mean(wr["k_copy"]["WRITE_SIZE"])
    ff, wf = copy_bytes / 1024 / fk, copy_bytes / 1024 / wk
    per = {}
    for k in fe:
        if k == "k_copy" or k not in wr:
            continue
        f, w = mean(fe[k]["FETCH_SIZE"]), mean(wr[k]["WRITE_SIZE"])
        per[k] = {"fetch_kib": f, "write_kib": w, "dispatches": len(fe[k]["FETCH_SIZE"]),
                  "hbm_bytes": (f * ff + w * wf) * 1024}
    cal = {"copy_bytes": copy_bytes, "fetch_kib_read": fk, "write_kib_read": wk, "fetch_factor": ff,
           "write_factor": wf}
    return cal, per


def table(rows, head, fmt):
    lines = [head]
    for r in rows:
        lines.append(fmt.format(*r))
    return "\n".join(lines)


def record_layer(d, out=PROFILES):
    bench = json.loads(open(os.path.join(d, "bench.json")).read().strip().splitlines()[-1])
    n, pairs = bench["config"]["active_sites"], bench["config"]["pairs"]
    cin, cout = bench["config"]["c_in"], bench["config"]["c_out"]
    sha = hashlib.sha256(open(KERNEL_SRC, "rb").read()).hexdigest()[:16]
    flops = 2.0 * cin * cout * pairs
    stats = kernel_stats(os.path.join(d, "trace"))
    dom = [r for r in stats if r[0] == DOMINANT]
    rof = bench["roofline"]

    # 1. kernel trace
    txt = [f"Kernel statistics: SSC 3^3 layer, 128^3 grid, batch 4, {n} surface sites, C_in = {cin}, "
           f"C_out = {cout}, {pairs} pairs",
           "(bench.py's layer workload: 13 steps incl. warmup, then its per-stage timing loops)", "",
           "Command (repo root, MI355X):", "  " + command("trace", "gpurun_out/prof"), "",
           f"conv.hip sha256[:16] = {sha}", ""]
    txt.append(table([(r[0][:62], r[1], r[2], r[3], r[4], r[5]) for r in stats if r[5] >= 0.3],
                     f"{'kernel':62s} {'calls':>6s} {'avg us':>9s} {'min us':>9s} {'max us':>9s} {'%':>6s}",
                     "{:62s} {:6d} {:9.2f} {:9.2f} {:9.2f} {:6.2f}"))
    if dom:
        avg = dom[0][2]
        txt += ["", f"Dominant kernel {DOMINANT} (the dgrad launch; k_conv_rows is the forward launch of the "
                    "same code):",
                f"  useful flops per launch 2 x {cin} x {cout} x {pairs} = {flops:.4g}",
                f"  rocprof average {avg:.2f} us -> {flops / (avg * 1e-6) / 1e12:.1f} TFLOP/s = "
                f"{flops / (avg * 1e-6) / 1e12 / 157.3:.3f} of 157.3",
                f"  bench.py's HIP-event mean of the same launches in this run: {rof['launch_ms'] * 1e3:.2f} us -> "
                f"frac {rof['frac']:.3f} (agreement {100 * (rof['launch_ms'] * 1e3 / avg - 1):+.1f}%)"]
    open(os.path.join(out, "k_dgrad_rows_ssc128_c64_kernel_stats.txt"), "w").write("\n".join(txt) + "\n")

    # 2. traffic record (read by bench.py)
    cal, per = calibrated_traffic(os.path.join(d, "fetch"), os.path.join(d, "write"))
    alg = {"X_read": n * cout * 4, "Y_write": n * cin * 4, "pair_rows_read": 8 * pairs, "W_read": 27 * cin * cout * 4}
    keep = {k: v for k, v in per.items() if v["hbm_bytes"] > 2e6}
    rec = {"kernel": DOMINANT, "workload": "ssc3x3x3_grid128_batch4_surfaces_c64", "source_sha256_16": sha,
           "fetch_cmd": command("fetch", "gpurun_out/prof"), "write_cmd": command("write", "gpurun_out/prof"),
           "summary_cmd": "python -m paper_1711_10275_amd.measure.record --dir gpurun_out/prof",
           "calibration": cal, "per_kernel": keep,
           "algorithmic_bytes_per_launch": alg, "algorithmic_bytes_total": sum(alg.values()),
           "hbm_bytes_per_launch": per[DOMINANT]["hbm_bytes"] if DOMINANT in per else None}
    json.dump(rec, open(os.path.join(out, "k_dgrad_rows_ssc128_c64_traffic.json"), "w"), indent=1)

    # 3. MFMA / LDS counters of the contraction kernels
    mf, ld = counters(os.path.join(d, "mfma")), counters(os.path.join(d, "lds"))
    durs = {r[0]: r[2] for r in stats}
    txt = ["MFMA and LDS counters of the contraction kernels, SSC 3^3 layer at 128^3 x 4 "
           f"({n} sites, {pairs} pairs, C = {cin}), fp32 and bf16 passes of bench.py",
           "", "Commands (repo root, MI355X; one counter pass per run):",
           "  " + command("mfma", "gpurun_out/prof"), "  " + command("lds", "gpurun_out/prof"), "",
           f"conv.hip sha256[:16] = {sha}", "",
           "busy = SQ_VALU_MFMA_BUSY_CYCLES / (1024 SIMDs x GRBM_GUI_ACTIVE / 8)  (the MFMA pipes' busy share)",
           "exec = 512 x (SQ_INSTS_VALU_MFMA_MOPS_BF16 + SQ_INSTS_VALU_MFMA_MOPS_F32), flops the MFMAs executed",
           f"useful = 2 x {cin} x {cout} x pairs = {flops:.4g} per launch; exec/useful counts the absent-neighbour",
           "  rows of the row blocks and, for fp32 through bf16 parts, the six bf16 products per fp32 product",
           "ldsconf = SQ_LDS_BANK_CONFLICT / SQ_ACTIVE_INST_LDS (bank-conflict cycles per LDS instruction cycle)", ""]
    rows = []
    for k in sorted(mf):
        if not ("rows" in k or "wgrad" in k):
            continue
        c = {x: mean(v) for x, v in mf[k].items()}
        l = {x: mean(v) for x, v in ld.get(k, {}).items()}
        cyc = c["GRBM_GUI_ACTIVE"] / N_XCD
        busy = c["SQ_VALU_MFMA_BUSY_CYCLES"] / (N_CU * SIMD_PER_CU * cyc)
        ex = 512.0 * (c.get("SQ_INSTS_VALU_MFMA_MOPS_BF16", 0) + c.get("SQ_INSTS_VALU_MFMA_MOPS_F32", 0))
        conf = l.get("SQ_LDS_BANK_CONFLICT", 0) / max(l.get("SQ_ACTIVE_INST_LDS", 1), 1)
        rows.append((k[:52], len(mf[k]["GRBM_GUI_ACTIVE"]), durs.get(k, float("nan")), busy, ex / 1e9,
                     ex / flops, conf))
    txt.append(table(rows, f"{'kernel':52s} {'disp':>5s} {'avg us':>8s} {'busy':>6s} {'exec GF':>8s} "
                           f"{'ex/use':>7s} {'ldsconf':>8s}",
                     "{:52s} {:5d} {:8.2f} {:6.3f} {:8.2f} {:7.2f} {:8.3f}"))
    txt += ["", "(avg us from the kernel trace of the same workload; the forward and dgrad launches of one",
            " dtype run the same code: k_conv_rows over the rule book, k_dgrad_rows over its transpose)"]
    open(os.path.join(out, "ssc128_c64_mfma_counters.txt"), "w").write("\n".join(txt) + "\n")


def record_all(d, out=PROFILES):
    b = json.loads(open(os.path.join(d, "bench_all.json")).read().strip().splitlines()[-1])
    stats = kernel_stats(os.path.join(d, "all"))
    e, u = b["extra"]["sc_then_ssc"], b["extra"]["unet"]
    txt = ["Kernel statistics of a whole bench.py run: the SSC 3^3 layer step (128^3 x 4 shapes, 100k sites, "
           "C = 64, fp32 and bf16),",
           "SC(2,2) 64 -> 96 then SSC 3^3 at 64^3 (fp32, bf16), and the five-level U-Net on 256^3 x 8 scenes "
           "(about 2M level-0",
           "sites, bf16, 32 -> 160 channels) with its geometry builds.", "",
           "Command (repo root, MI355X):", "  " + command("all", "gpurun_out/prof"), "",
           "bench.py's own figures from this profiled run (the profiler's per-dispatch cost inflates short "
           "launches and host-bound phases):",
           f"  layer step {b['ms_per_step']:.3f} ms; dgrad row launch {b['roofline']['launch_ms'] * 1e3:.1f} us "
           f"(frac {b['roofline']['frac']:.3f})",
           f"  U-Net forward {u['forward_ms']:.3f} ms = {u['forward_effective_tflops']:.0f} effective TFLOP/s "
           f"({u['flops']:.4g} flops), unfused heads {u['forward_unfused_ms']:.3f} ms",
           f"  U-Net geometry (all rule books + plans) {u['geometry_build_ms']:.3f} ms; fresh input (geometry + "
           f"forward) {u['geometry_plus_forward_ms']:.3f} ms",
           f"  level-0 SSC build {u['level0_ssc_build_roofline']['ms']:.3f} ms; level sites {u['level_sites']}",
           f"  SC(2,2) forward fp32 {e['sc_forward_ms_f32'] * 1e3:.1f} us, bf16 {e['sc_forward_ms_bf16'] * 1e3:.1f} "
           f"us; SSC 64^3 C=96 fp32 {e['ssc_forward_ms_f32'] * 1e3:.1f} us, bf16 "
           f"{e['ssc_forward_ms_bf16'] * 1e3:.1f} us", ""]
    o = b["extra"].get("ops")
    if o:
        f = lambda d: f"{d['ms'] * 1e3:.1f} us ({100 * d['frac']:.0f}% of HBM)"
        pl, bn = o["pool"]["f32"], o["batchnorm"]["scenes256_c32_bf16"]
        txt += [f"  MP forward / backward (SC(2,2), C = 64 fp32) {f(pl['max_forward'])} / {f(pl['max_backward'])}; "
                f"upsampling {f(pl['upsample_forward'])}",
                f"  BN at 2M x 32 bf16: statistics {f(bn['stats'])}, apply {f(bn['apply_relu'])}, parameter "
                f"gradients {f(bn['backward_params'])}, input gradient {f(bn['backward_input'])}",
                f"  U-Net training step (256^3 x 8, bf16) {o['unet_train_step']['ms']:.2f} ms; residual block "
                f"forward {o['residual_block']['forward_ms'] * 1e3:.0f} us; 4-d SSC(3) layer forward "
                f"{o['layer_4d']['forward_ms'] * 1e3:.0f} us", ""]
    tot = sum(r[1] * r[2] for r in stats)
    rows = [(r[0][:64], r[1], r[2], r[1] * r[2] / 1e3, r[5]) for r in stats if r[5] >= 0.25]
    txt.append(table(rows, f"{'kernel (all launches of the run)':64s} {'calls':>6s} {'avg us':>9s} "
                           f"{'total ms':>9s} {'%':>6s}", "{:64s} {:6d} {:9.2f} {:9.3f} {:6.2f}"))
    txt.append(f"(kernels under 0.25% not listed; all kernels together {tot / 1e3:.1f} ms)")
    open(os.path.join(out, "bench_all_workloads_kernel_stats.txt"), "w").write("\n".join(txt) + "\n")


def record_builds(d, out=PROFILES):
    b = json.loads(open(os.path.join(d, "builds.json")).read().strip().splitlines()[-1])
    stats = kernel_stats(os.path.join(d, "btrace"))
    cal, per = calibrated_traffic(os.path.join(d, "bfetch"), os.path.join(d, "bwrite"))
    txt = [f"Rule-book builds at {b['sites']} sites (256^3 x 8 scenes): SSC 3^3 ({b['ssc_pairs']} pairs) and "
           f"SC(2,2) ({b['sc_out_sites']} output sites, {b['sc_pairs']} pairs)",
           f"wall time per build under the kernel-trace profiler: SSC {b['ssc_build_ms']:.3f} ms, "
           f"SC {b['sc_build_ms']:.3f} ms", "",
           "Commands (repo root, MI355X):"] + ["  " + command(p, "gpurun_out/prof") for p in ("btrace", "bfetch",
                                                                                            "bwrite")]
    txt += ["", f"calibration (256 MiB copy): fetch x{cal['fetch_factor']:.3f}, write x{cal['write_factor']:.3f}",
            "", ]
    rows = []
    for r in stats:
        if r[0] in ("k_copy",) or r[5] < 0.2:
            continue
        t = per.get(r[0])
        rows.append((r[0][:40], r[1], r[2], (t["fetch_kib"] * cal["fetch_factor"] * 1024 / 1e6) if t else float("nan"),
                     (t["write_kib"] * cal["write_factor"] * 1024 / 1e6) if t else float("nan")))
    txt.append(table(rows, f"{'kernel':40s} {'calls':>6s} {'avg us':>9s} {'fetch MB':>9s} {'write MB':>9s}",
                     "{:40s} {:6d} {:9.2f} {:9.2f} {:9.2f}"))
    open(os.path.join(out, "rulebook_build_scenes256_traffic.txt"), "w").write("\n".join(txt) + "\n")


def main():
    p = argparse.ArgumentParser()
    p.add_argument("--dir", help="rocprofv3 output of the passes")
    p.add_argument("--show-commands", metavar="DIR", help="print the passes' commands, writing under DIR")
    p.add_argument("--out", default=PROFILES, help="where the summaries go")
    a = p.parse_args()
    if a.show_commands:
        for name in PASSES:
            print(command(name, a.show_commands))
        return
    record_layer(a.dir, a.out)
    record_all(a.dir, a.out)
    record_builds(a.dir, a.out)


if __name__ == "__main__":
    main()
