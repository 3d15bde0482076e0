"""Benchmark of the SSC 3^3 layer hot path on one MI355X.

Workload: 128^3 grid, batch 4, each sample the union of 8 seeded random
surfaces (sphere shells, planar patches, cylinder shells) voxelised to a
1-voxel-thick surface, about 100k active sites; C_in = C_out = 64, fp32.
Features N(0,1), weights N(0, 1/(27 C_in)), upstream gradient N(0,1).

One step = rule-book build (dictionary, neighbour probe, compaction, the
row-block plan, one readback) + forward + dgrad (over the transposed rule
book) + wgrad (per offset): every stage of the layer.  Inputs are resident
in HBM before the timed region.  value = active sites / s over whole steps.

Dominant kernel: the row-block kernel, launched once by the forward
(k_conv_rows) and once by the dgrad (k_dgrad_rows, the same code under its
own name).  Its duration is measured inside the timed steps: before each
step's backward call the library is asked (sscn_time_next_launch) to
record a pair of HIP events around its next row-block launch, which is the
dgrad kernel, on its stream (the small weight-split kernel queued before it
stays outside the pair); `roofline` divides the useful flops of one launch
(2 C_in C_out per pair, Table 2) by the mean of those durations.  `traffic` (HBM bytes per launch) comes from
the committed counter record in profiles/ and is null when the kernel
source has changed since those counters were taken.  `build_roofline` puts
the SSC build's algorithmic bytes over its wall time against HBM bandwidth;
the builder's own intermediate (its neighbour map, written and read back)
is reported beside them and not counted.

Also reported: per-stage times (fp32 and bf16), a cold-cache step (after a
512 MB flush write), the same layer with its rows shuffled (locality), the
measured ceilings of the box (a streaming copy and register-only MFMA
loops), and the CPU oracle timed on a bounded sample of the same workload
on the host cores.

--copy-calibration runs a plain 256 MiB device copy (the measure library's
k_copy) so that a counter run can scale FETCH_SIZE / WRITE_SIZE by what
they read for it.
"""
from __future__ import annotations

import argparse
import ctypes
import hashlib
import json
import os
import platform
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_FP32_MFMA_TFLOPS = 157.3
PEAK_BF16_MFMA_TFLOPS = 2500.0
PEAK_HBM_GBS = 8000.0
METRIC = "SSC 3^3 layer active-sites/s + effective TFLOP/s; rulebook build ms"
KERNEL_SRC = os.path.join(ROOT, "paper_1711_10275_amd", "csrc", "conv.hip")
TRAFFIC_RECORD = os.path.join(ROOT, "profiles", "k_dgrad_rows_ssc128_c64_traffic.json")
DOMINANT = "k_dgrad_rows<float, 128, 4, 2, 1, false, true>"
MEASURE_LIB = os.path.join(ROOT, "paper_1711_10275_amd", "libsscn_measure.so")


def kernel_source_hash():
    return hashlib.sha256(open(KERNEL_SRC, "rb").read()).hexdigest()[:16]


def recorded_traffic():
    """HBM bytes per launch of the dominant kernel from the committed counter
    record, if it was taken on the current kernel source."""
    try:
        rec = json.load(open(TRAFFIC_RECORD))
    except (OSError, ValueError):
        return None
    if rec.get("source_sha256_16") != kernel_source_hash():
        return None
    return rec.get("hbm_bytes_per_launch")


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=20)
    p.add_argument("--warmup", type=int, default=5)
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--cpu-seconds", type=float, default=12.0, help="bound on the CPU oracle sample")
    p.add_argument("--copy-calibration", action="store_true",
                   help="also run a 256 MiB device copy (counter calibration)")
    p.add_argument("--no-extra", action="store_true",
                   help="skip the SC -> SSC, U-Net, cold-cache, shuffled and ceiling figures")
    return p.parse_args()


def host_cpu():
    model = platform.processor() or "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return model, os.cpu_count()


def cpu_baseline(coords, size, X, W, G, budget_s):
    """The oracle as it stands, timed on whole steps of the same workload."""
    from oracle import sscn_oracle as O
    try:
        import threadpoolctl
        threads = max([i.get("num_threads", 1) for i in threadpoolctl.threadpool_info()] or [1])
    except Exception:
        threads = 1
    n = coords.shape[0]
    steps, t_total = 0, 0.0
    while t_total < budget_s and steps < 20:
        t0 = time.perf_counter()
        orb = O.ssc_rulebook(coords, size, 3)
        O.forward(X, W, orb)
        O.backward(X, W, G, orb)
        t_total += time.perf_counter() - t0
        steps += 1
    model, ncpu = host_cpu()
    return {"value": n * steps / t_total, "unit": "active-sites/s", "cores": int(threads), "kind": "oracle",
            "host_cpus": ncpu, "cpu_model": model,
            "sample": f"{steps} whole steps (rule book + forward + backward, numpy fp64; its matrix products "
                      f"use {threads} BLAS threads, the rest one) of the same {n}-site workload, {t_total:.1f} s"}


def _event_ms(fn, reps, stream):
    """Mean time per call of back-to-back calls (HIP events on `stream`)."""
    import torch
    fn()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(reps):
        fn()
    e1.record(stream)
    e1.synchronize()
    return e0.elapsed_time(e1) / reps


def _wall_ms(fn, reps):
    import torch
    fn()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(reps):
        fn()
    torch.cuda.synchronize()
    return (time.perf_counter() - t0) * 1e3 / reps


def table_capacity(n):
    cap = 64
    while cap < 2 * n:
        cap *= 2
    return cap


def build_roofline(n, K, pairs, ms, what, slot=8):
    """Algorithmic bytes of an SSC rule-book build against HBM bandwidth.

    Counted: coordinates read (16 B per site), the dictionary filled and its
    slots written (slot bytes each: 8 for the 32-bit keys that both
    workloads here use; capacity the power of two >= 2n), one slot read per
    lookup performed (K per site below 2^18 sites; from 2^18 the mirrored
    probe looks up only the (K - 1) / 2 offsets below the centre and derives
    the rest), and the pair arrays written (8 B per pair).  Not counted: the
    builder's neighbour map (4 B per site and offset, written and read back),
    reported as `intermediate_bytes`.  The time is the host wall time of the
    build call (its row-block plan and readback included).
    """
    cap = table_capacity(n)
    lookups = K * n if n < (1 << 18) else (K - 1) // 2 * n
    nbytes = 16 * n + 2 * slot * cap + slot * lookups + 8 * pairs
    achieved = nbytes / (ms * 1e-3) / 1e9
    return {"stage": what, "bound": "hbm", "achieved": achieved, "peak": PEAK_HBM_GBS, "unit": "GB/s",
            "frac": achieved / PEAK_HBM_GBS, "bytes": nbytes, "ms": ms, "intermediate_bytes": 8 * K * n}


def measured_ceilings():
    """Copy bandwidth and MFMA-loop rates measured on this GPU."""
    L = ctypes.CDLL(MEASURE_LIB)
    L.sscn_measure_copy.argtypes = [ctypes.c_int64, ctypes.c_int, ctypes.POINTER(ctypes.c_double)]
    L.sscn_measure_mfma.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.POINTER(ctypes.c_double)]
    out = {}
    v = ctypes.c_double()
    if L.sscn_measure_copy(1 << 30, 5, ctypes.byref(v)) == 0:
        out["copy_1GiB_GBs"] = v.value
    if L.sscn_measure_mfma(0, 5, ctypes.byref(v)) == 0:
        out["mfma_f32_16x16x4_TFLOPs"] = v.value
    if L.sscn_measure_mfma(1, 5, ctypes.byref(v)) == 0:
        out["mfma_bf16_16x16x32_TFLOPs"] = v.value
    return out


def copy_calibration():
    L = ctypes.CDLL(MEASURE_LIB)
    L.sscn_measure_copy.argtypes = [ctypes.c_int64, ctypes.c_int, ctypes.POINTER(ctypes.c_double)]
    v = ctypes.c_double()
    L.sscn_measure_copy(256 << 20, 2, ctypes.byref(v))


def sc_then_ssc(tc, size, stream, reps):
    """SC(2, 2) 64 -> 96 channels (128^3 -> 64^3), then SSC 3^3 at 64^3 with 96 channels."""
    import torch
    from paper_1711_10275_amd import sscn
    from paper_1711_10275_amd import synthetic as S
    dev = tc.device
    sc_build = _wall_ms(lambda: sscn.sc_rulebook_build(tc, size, 2, 2), reps)
    sc = sscn.sc_rulebook_build(tc, size, 2, 2)
    oc = sc.out_coords()
    ssc_build = _wall_ms(lambda: sscn.ssc_rulebook_build(oc, sc.out_size, 3), reps)
    ssc = sscn.ssc_rulebook_build(oc, sc.out_size, 3)
    out = {"workload": "sc2x2x2s2_grid128to64_c64to96_then_ssc3x3x3_grid64_c96", "sc_out_sites": sc.n_out,
           "sc_pairs": sc.n_pairs, "ssc_pairs": ssc.n_pairs, "sc_rulebook_build_ms": sc_build,
           "ssc_rulebook_build_ms": ssc_build}
    for name, dt in (("f32", torch.float32), ("bf16", torch.bfloat16)):
        X = torch.from_numpy(S.features(tc.shape[0], 64, S.SEED_FEAT + 2)).to(dt).to(dev)
        W1 = torch.from_numpy(S.weights(8, 64, 96, S.SEED_WEIGHT + 2)).to(dt).to(dev)
        W2 = torch.from_numpy(S.weights(27, 96, 96, S.SEED_WEIGHT + 22)).to(dt).to(dev)
        Y = sscn.sparse_conv_forward(X, W1, sc)
        t1 = _event_ms(lambda: sscn.sparse_conv_forward(X, W1, sc), reps, stream)
        t2 = _event_ms(lambda: sscn.sparse_conv_forward(Y, W2, ssc), reps, stream)
        out[f"sc_forward_ms_{name}"] = t1
        out[f"ssc_forward_ms_{name}"] = t2
        out[f"sc_tflops_{name}"] = 2.0 * 64 * 96 * sc.n_pairs / (t1 * 1e-3) / 1e12
        out[f"ssc_tflops_{name}"] = 2.0 * 96 * 96 * ssc.n_pairs / (t2 * 1e-3) / 1e12
    return out


def unet_scenes(stream, reps):
    """Five-level submanifold U-Net forward, 256^3 x 8 scenes, bf16."""
    import torch
    from paper_1711_10275_amd import sscn, unet
    from paper_1711_10275_amd import synthetic as S
    dev = torch.device("cuda:0")
    c = S.scenes_256()
    tc = torch.from_numpy(c).to(dev)
    X = torch.from_numpy(S.features(c.shape[0], 32, S.SEED_FEAT + 3, bf16=True)).to(torch.bfloat16).to(dev)
    params = unet.device_params(draw=lambda n, k, ci, co: S.layer_params(n, k, ci, co, bf16=True))
    geom_ms = _wall_ms(lambda: unet.Geometry(tc, (256, 256, 256)), reps)
    ssc0_ms = _wall_ms(lambda: sscn.ssc_rulebook_build(tc, (256, 256, 256), 3), reps)
    ssc0_pairs = sscn.ssc_rulebook_build(tc, (256, 256, 256), 3).n_pairs
    # a fresh input: rule books of every level, then the network (lazily built
    # tables included)
    fresh_ms = _wall_ms(lambda: unet.forward(X, unet.Geometry(tc, (256, 256, 256)), params), reps)
    geom = unet.Geometry(tc, (256, 256, 256))
    fwd_ms = _event_ms(lambda: unet.forward(X, geom, params), reps, stream)
    unfused_ms = _event_ms(lambda: unet.forward(X, geom, params, fused=False), reps, stream)
    fl = unet.flops(geom)
    return {"workload": "unet5_grid256_batch8_scenes_c32to160_bf16", "level_sites": [int(x.shape[0]) for x in geom.coords],
            "geometry_build_ms": geom_ms,
            "level0_ssc_build_roofline": build_roofline(int(c.shape[0]), 27, int(ssc0_pairs), ssc0_ms,
                                                        "SSC 3^3 rule-book build incl. its row-block plan, "
                                                        "level 0 (about 2M sites)"),
            "forward_ms": fwd_ms, "forward_sites_per_s": c.shape[0] / (fwd_ms * 1e-3),
            "forward_effective_tflops": fl / (fwd_ms * 1e-3) / 1e12, "flops": fl,
            "forward_unfused_ms": unfused_ms, "geometry_plus_forward_ms": fresh_ms,
            "geometry_plus_forward_sites_per_s": c.shape[0] / (fresh_ms * 1e-3)}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for {args.gpus}); the layer is not sharded across GPUs.",
              file=sys.stderr)
        sys.exit(2)
    import torch
    from paper_1711_10275_amd import sscn
    from paper_1711_10275_amd import synthetic as S

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    coords = S.shapes_128()
    size = (128, 128, 128)
    n, cin, cout = coords.shape[0], 64, 64
    X = S.features(n, cin, S.SEED_FEAT + 1)
    W = S.weights(27, cin, cout, S.SEED_WEIGHT + 1)
    G = S.features(n, cout, S.SEED_GRAD + 1)
    tc = torch.from_numpy(coords).to(dev)
    tX, tW, tG = (torch.from_numpy(a).to(dev) for a in (X, W, G))
    stream = torch.cuda.current_stream(dev)
    timers = [sscn.KernelTimer() for _ in range(args.steps)]

    def step(tc=tc, tX=tX, tG=tG, timer=None):
        rb = sscn.ssc_rulebook_build(tc, size, 3)
        sscn.sparse_conv_forward(tX, tW, rb)
        if timer is not None:
            timer.arm()  # the backward's first row-block launch: the dgrad kernel
        sscn.sparse_conv_backward(tX, tW, tG, rb)
        return rb

    for _ in range(args.warmup):
        rb = step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        rb = step(timer=timers[i])
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms_step = (t1 - t0) * 1e3 / args.steps
    launch_ms = sum(t.ms() for t in timers) / len(timers)
    pairs = rb.n_pairs
    flops_layer = 2.0 * cin * cout * pairs  # useful flops of one pass (fwd, dgrad or wgrad)

    # ---- per-stage breakdown (same stream; events bracket the calls) ----
    reps = max(10, args.steps)
    torch.cuda.synchronize()
    tb = time.perf_counter()
    for _ in range(reps):
        rbx = sscn.ssc_rulebook_build(tc, size, 3)
    torch.cuda.synchronize()
    build_ms = (time.perf_counter() - tb) * 1e3 / reps
    del rbx

    timed = lambda fn: _event_ms(fn, reps, stream)
    fwd_ms = timed(lambda: sscn.sparse_conv_forward(tX, tW, rb))
    dgrad_ms = timed(lambda: sscn.sparse_conv_backward(None, tW, tG, rb, dgrad=True, wgrad=False))
    if args.copy_calibration:
        copy_calibration()
    wgrad_ms = timed(lambda: sscn.sparse_conv_backward(tX, tW, tG, rb, dgrad=False, wgrad=True))
    tXb, tWb, tGb = tX.to(torch.bfloat16), tW.to(torch.bfloat16), tG.to(torch.bfloat16)
    fwd_bf16_ms = timed(lambda: sscn.sparse_conv_forward(tXb, tWb, rb))
    dgrad_bf16_ms = timed(lambda: sscn.sparse_conv_backward(None, tWb, tGb, rb, dgrad=True, wgrad=False))
    wgrad_bf16_ms = timed(lambda: sscn.sparse_conv_backward(tXb, tWb, tGb, rb, dgrad=False, wgrad=True))

    achieved = flops_layer / (launch_ms * 1e-3) / 1e12
    result = {
        "metric": METRIC,
        "value": n / (ms_step * 1e-3),
        "unit": "active-sites/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": "ssc3x3x3_grid128_batch4_surfaces_c64", "active_sites": int(n),
                   "pairs": int(pairs), "c_in": cin, "c_out": cout,
                   "step": "rule-book build + forward + backward (dgrad + wgrad)"},
        "effective_tflops_step": 3 * flops_layer / (ms_step * 1e-3) / 1e12,
        "rulebook_build_ms": build_ms,
        "forward_ms": fwd_ms,
        "forward_tflops": flops_layer / (fwd_ms * 1e-3) / 1e12,
        "forward_sites_per_s": n / (fwd_ms * 1e-3),
        "dgrad_ms": dgrad_ms,
        "wgrad_ms": wgrad_ms,
        "wgrad_tflops": flops_layer / (wgrad_ms * 1e-3) / 1e12,
        "bf16": {"forward_ms": fwd_bf16_ms, "dgrad_ms": dgrad_bf16_ms, "wgrad_ms": wgrad_bf16_ms,
                 "forward_tflops": flops_layer / (fwd_bf16_ms * 1e-3) / 1e12},
        "roofline": {"kernel": DOMINANT + " (the dgrad launch of the row-block kernel; the forward launches "
                               "the same code as k_conv_rows; fp32 through three bf16 parts on 16x16x32 MFMAs)",
                     "bound": "mfma", "achieved": achieved, "peak": PEAK_FP32_MFMA_TFLOPS,
                     "unit": "TFLOP/s", "frac": achieved / PEAK_FP32_MFMA_TFLOPS,
                     "launch_ms": launch_ms, "launches_timed": len(timers),
                     "flops_per_launch": flops_layer, "traffic": recorded_traffic()},
        "build_roofline": build_roofline(int(n), 27, int(pairs), build_ms,
                                         "SSC 3^3 rule-book build incl. its row-block plan, 100k sites"),
    }
    if not args.no_extra:
        ceil = measured_ceilings()
        result["measured_ceilings"] = ceil
        if "mfma_f32_16x16x4_TFLOPs" in ceil:
            result["roofline"]["peak_measured"] = ceil["mfma_f32_16x16x4_TFLOPs"]
            result["roofline"]["frac_of_measured"] = achieved / ceil["mfma_f32_16x16x4_TFLOPs"]
        if "copy_1GiB_GBs" in ceil:
            result["build_roofline"]["peak_measured"] = ceil["copy_1GiB_GBs"]
        # cold caches: a 512 MB write evicts the 256 MB last-level cache before one step
        flush = torch.empty(128 << 20, dtype=torch.float32, device=dev)
        cold = []
        for _ in range(3):
            flush.fill_(1.0)
            torch.cuda.synchronize()
            tcold = time.perf_counter()
            step()
            torch.cuda.synchronize()
            cold.append((time.perf_counter() - tcold) * 1e3)
        del flush
        result["cold_step_ms"] = float(np.median(cold))
        # locality: the same sites with their rows shuffled
        perm_coords = S.shuffled(coords, 77)
        tcs = torch.from_numpy(perm_coords).to(dev)
        shuffled_ms = _wall_ms(lambda: step(tc=tcs), reps)
        rbs = sscn.ssc_rulebook_build(tcs, size, 3)
        result["shuffled_rows"] = {"step_ms": shuffled_ms,
                                   "forward_ms": timed(lambda: sscn.sparse_conv_forward(tX, tW, rbs)),
                                   "dgrad_ms": timed(lambda: sscn.sparse_conv_backward(None, tW, tG, rbs, wgrad=False))}
        del rbs
        result["extra"] = {"sc_then_ssc": sc_then_ssc(tc, size, stream, reps), "unet": unet_scenes(stream, 5)}
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(coords, size, X, W, G, args.cpu_seconds)
    print(json.dumps(result))


if __name__ == "__main__":
    main()
