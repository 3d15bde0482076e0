"""Benchmark of the SSC 3^3 layer hot path on one MI355X.

Workload: 128^3 grid, batch 4, each sample the union of 8 seeded random
surfaces (sphere shells, planar patches, cylinder shells) voxelised to a
1-voxel-thick surface, about 100k active sites; C_in = C_out = 64, fp32.
Features N(0,1), weights N(0, 1/(27 C_in)), upstream gradient N(0,1).

One step = rule-book build (dictionary, neighbour probe, compaction, one
readback) + forward + backward (dgrad over the transposed rule book, wgrad
per offset): every stage of the layer.  Inputs are resident in HBM before
the timed region.  value = active sites / s over whole steps.

Also reported: per-stage times, useful ("effective") TFLOP/s counting only
the multiply-adds of real pairs (2 C_in C_out per pair, Table 2), the
roofline of the dominant kernel and the CPU oracle timed on a bounded
sample of the same workload on the host cores.

Dominant kernel: k_conv_quad, which runs the forward and the dgrad of the
layer (same pairs, same channel counts).  Its duration is measured with HIP
events around the dgrad call, which is exactly one launch of it on the
current stream.  `traffic` (HBM bytes per launch) comes from the committed
counter record in profiles/, and is null when the kernel source has changed
since those counters were taken.

--copy-calibration runs a plain device copy of known size (256 MiB) so
that a counter run can scale FETCH_SIZE / WRITE_SIZE by what they read for
it.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
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
TRAFFIC_RECORD = os.path.join(ROOT, "profiles", "k_conv_quad_ssc128_c64_traffic.json")


def kernel_source_hash():
    return hashlib.sha256(open(KERNEL_SRC, "rb").read()).hexdigest()[:16]


def recorded_traffic():
    """HBM bytes per launch from the committed counter record, if still valid."""
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
    return p.parse_args()


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
    return {"value": n * steps / t_total, "unit": "active-sites/s", "cores": int(threads), "kind": "oracle",
            "sample": f"{steps} whole steps (rule book + forward + backward, numpy fp64) of the same "
                      f"{n}-site workload, {t_total:.1f} s"}


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

    def step():
        rb = sscn.ssc_rulebook_build(tc, size, 3)
        sscn.sparse_conv_forward(tX, tW, rb)
        sscn.sparse_conv_backward(tX, tW, tG, rb)
        return rb

    for _ in range(args.warmup):
        rb = step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        rb = step()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms_step = (t1 - t0) * 1e3 / args.steps
    pairs = rb.n_pairs
    flops_layer = 2.0 * cin * cout * pairs  # useful flops of one pass (fwd, dgrad or wgrad)

    # ---- per-stage breakdown (same stream; events bracket the calls) ----
    stream = torch.cuda.current_stream(dev)
    reps = max(10, args.steps)
    torch.cuda.synchronize()
    tb = time.perf_counter()
    for _ in range(reps):
        rbx = sscn.ssc_rulebook_build(tc, size, 3)
    torch.cuda.synchronize()
    build_ms = (time.perf_counter() - tb) * 1e3 / reps
    del rbx

    def timed(fn):
        fn()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(reps):
            fn()
        e1.record(stream)
        e1.synchronize()
        return e0.elapsed_time(e1) / reps

    fwd_ms = timed(lambda: sscn.sparse_conv_forward(tX, tW, rb))
    dgrad_ms = timed(lambda: sscn.sparse_conv_backward(None, tW, tG, rb, dgrad=True, wgrad=False))
    if args.copy_calibration:
        src = torch.empty(64 << 20, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
    wgrad_ms = timed(lambda: sscn.sparse_conv_backward(tX, tW, tG, rb, dgrad=False, wgrad=True))
    tXb, tWb = tX.to(torch.bfloat16), tW.to(torch.bfloat16)
    fwd_bf16_ms = timed(lambda: sscn.sparse_conv_forward(tXb, tWb, rb))

    achieved = flops_layer / (dgrad_ms * 1e-3) / 1e12  # one launch of the dominant kernel
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
        "forward_bf16_ms": fwd_bf16_ms,
        "forward_bf16_tflops": flops_layer / (fwd_bf16_ms * 1e-3) / 1e12,
        "roofline": {"kernel": "k_conv_quad<float> (forward/dgrad main kernel; timed on the dgrad call)",
                     "bound": "mfma", "achieved": achieved, "peak": PEAK_FP32_MFMA_TFLOPS,
                     "unit": "TFLOP/s", "frac": achieved / PEAK_FP32_MFMA_TFLOPS,
                     "launch_ms": dgrad_ms, "flops_per_launch": flops_layer,
                     "traffic": recorded_traffic()},
    }
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(coords, size, X, W, G, args.cpu_seconds)
    print(json.dumps(result))


if __name__ == "__main__":
    main()
