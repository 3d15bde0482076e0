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


def cpu_ops(coords, size):
    """The oracle on the further operators (pooling, batch normalisation, a
    residual block, a small U-Net training step, a 4-d layer), one timed
    call each, on the host cores: the CPU figures beside ops_extra's."""
    from oracle import sscn_oracle as O
    from paper_1711_10275_amd import synthetic as S
    from paper_1711_10275_amd import unet

    def t(fn):
        t0 = time.perf_counter()
        fn()
        return (time.perf_counter() - t0) * 1e3

    out = {}
    n = coords.shape[0]
    sc = O.sc_rulebook(coords, size, 2, 2)
    X = S.features(n, 64, S.SEED_FEAT + 41)
    out["max_pool_forward_ms"] = t(lambda: O.max_pool(X, sc))
    out["avg_pool_forward_ms"] = t(lambda: O.avg_pool(X, sc))
    g, b = np.ones(64), np.zeros(64)
    Y, mean, var = O.batch_norm_relu_train(X, g, b)
    out["batchnorm_forward_shapes128_c64_ms"] = t(lambda: O.batch_norm_relu_train(X, g, b))
    out["batchnorm_backward_shapes128_c64_ms"] = t(lambda: O.batch_norm_relu_backward(Y, X, g, b, mean, var))
    rb = O.ssc_rulebook(coords, size, 3)
    ps = [S.layer_params(f"res{i}", 27, 64, 64, bf16=False) for i in range(2)]
    out["residual_block_forward_ms"] = t(lambda: O.residual_block(X, rb, ps[0], ps[1]))
    cs = S.scenes_small(batch=2, L=32, target_per_sample=3000)
    ch, ncls = (8, 16, 24), 6
    Xs = S.features(cs.shape[0], ch[0], S.SEED_FEAT + 31)
    lab = S.labels(cs.shape[0], ncls, 32)
    out["unet3_train_step_scenes32_ms"] = t(lambda: O.unet_train_step(cs, (32, 32, 32), Xs, lab,
                                                                       lambda nm, k, ci, co: S.train_params(nm, k, ci,
                                                                                                            co),
                                                                       ch, ncls))
    out["unet3_train_step_scenes32_sites"] = int(cs.shape[0])
    c4 = S.moving_shells_4d()
    out["layer_4d_rulebook_ms"] = t(lambda: O.ssc_rulebook(c4, (16, 48, 48, 48), 3))
    r4 = O.ssc_rulebook(c4, (16, 48, 48, 48), 3)
    X4, W4 = S.features(c4.shape[0], 32, S.SEED_FEAT + 47), S.weights(81, 32, 32, S.SEED_WEIGHT + 47)
    out["layer_4d_forward_ms"] = t(lambda: O.forward(X4, W4, r4))
    return out


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


def _latency_ms(fn, reps):
    """Mean host time of single calls, each started on an idle GPU."""
    import torch
    fn()
    torch.cuda.synchronize()
    total = 0.0
    for _ in range(reps):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        r = fn()
        total += time.perf_counter() - t0
        del r
    torch.cuda.synchronize()
    return total * 1e3 / reps


def table_capacity(n):
    cap = 64
    while cap < 2 * n:
        cap *= 2
    return cap


def build_roofline(n, K, pairs, ms, what, slot=16, pairs_ms=None):
    """Algorithmic bytes of an SSC rule-book build against HBM bandwidth.

    Counted: coordinates read (16 B per site), the dictionary filled (slot
    bytes per slot: 16 for the grouped slots of the 32-bit keys that both
    workloads here use; capacity the power of two >= 2n slots), the inserts
    (a group key and a row, 8 B per site), the two words (8 B) read per
    lookup performed (K per site below 2^18 sites; from 2^18 the mirrored
    probe looks up only the (K - 1) / 2 offsets below the centre and derives
    the rest), and the pair arrays written (8 B per pair).  Not counted: the
    builder's neighbour map (4 B per site and offset, written and read back),
    reported as `intermediate_bytes`.  The time is the mean host wall time
    of back-to-back build calls: each call waits for its own readback of
    sizes and flags, and the row-block plan it queues behind that readback
    runs before the next call's kernels.  `pairs_ms` (if given) is the
    latency of one call on an idle GPU, until the pair arrays, sizes and
    flags are ready (the plan runs after the call returns): the time of the
    rule book the counted bytes belong to, reported as `rulebook_ms` with
    its own fraction `frac_rulebook`.
    """
    cap = table_capacity(n)
    lookups = K * n if n < (1 << 18) else (K - 1) // 2 * n
    nbytes = 16 * n + slot * cap + 8 * n + 8 * lookups + 8 * pairs
    achieved = nbytes / (ms * 1e-3) / 1e9
    out = {"stage": what, "bound": "hbm", "achieved": achieved, "peak": PEAK_HBM_GBS, "unit": "GB/s",
           "frac": achieved / PEAK_HBM_GBS, "bytes": nbytes, "ms": ms, "intermediate_bytes": 8 * K * n}
    if pairs_ms is not None:
        out["rulebook_ms"] = pairs_ms
        out["frac_rulebook"] = nbytes / (pairs_ms * 1e-3) / 1e9 / PEAK_HBM_GBS
    return out


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


def scaling_in_sites(stream, reps):
    """Cost against the number of active sites (the paper's O(a) per layer):
    the SSC 3^3 rule-book build and the fp32 64-channel forward on the
    1.8k-site shell (32^3), the 100k-site shapes (128^3 x 4) and the 2M-site
    scenes (256^3 x 8)."""
    import torch
    from paper_1711_10275_amd import sscn
    from paper_1711_10275_amd import synthetic as S
    out = []
    for name, coords, size in (("shell32", S.shell_32(), (32,) * 3), ("shapes128", S.shapes_128(), (128,) * 3),
                               ("scenes256", S.scenes_256(), (256,) * 3)):
        tc = torch.from_numpy(coords).cuda()
        n = int(coords.shape[0])
        build_ms = _wall_ms(lambda: sscn.ssc_rulebook_build(tc, size, 3), reps)
        rb = sscn.ssc_rulebook_build(tc, size, 3)
        X = torch.from_numpy(S.features(n, 64, S.SEED_FEAT + 5)).cuda()
        W = torch.from_numpy(S.weights(27, 64, 64, S.SEED_WEIGHT + 5)).cuda()
        fwd_ms = _event_ms(lambda: sscn.sparse_conv_forward(X, W, rb), reps, stream)
        out.append({"set": name, "sites": n, "pairs": int(rb.n_pairs), "rulebook_build_ms": build_ms,
                    "build_us_per_1k_sites": build_ms * 1e3 / (n / 1e3), "forward_ms_f32_c64": fwd_ms,
                    "forward_sites_per_s": n / (fwd_ms * 1e-3),
                    "forward_tflops": 2.0 * 64 * 64 * rb.n_pairs / (fwd_ms * 1e-3) / 1e12})
        del rb, X, W, tc
    return out


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
    ssc0_lat = _latency_ms(lambda: sscn.ssc_rulebook_build(tc, (256, 256, 256), 3), reps)
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
                                                        "level 0 (about 2M sites)", pairs_ms=ssc0_lat),
            "forward_ms": fwd_ms, "forward_sites_per_s": c.shape[0] / (fwd_ms * 1e-3),
            "forward_effective_tflops": fl / (fwd_ms * 1e-3) / 1e12, "flops": fl,
            "forward_unfused_ms": unfused_ms, "geometry_plus_forward_ms": fresh_ms,
            "geometry_plus_forward_sites_per_s": c.shape[0] / (fresh_ms * 1e-3)}


def _hbm(nbytes, ms):
    gbs = nbytes / (ms * 1e-3) / 1e9
    return {"ms": ms, "bytes": int(nbytes), "achieved_GBs": gbs, "peak_GBs": PEAK_HBM_GBS, "frac": gbs / PEAK_HBM_GBS}


def ops_extra(tc, size, stream, reps):
    """The operators beyond the convolution (pooling, upsampling, batch
    normalisation, the training step, residual blocks, bias, 4-d layers),
    each timed with its algorithmic bytes (HBM-bound operators) or useful
    flops (convolutions) against the peak."""
    import torch
    from paper_1711_10275_amd import blocks, sscn, train, unet
    from paper_1711_10275_amd import synthetic as S
    dev = tc.device
    timed = lambda fn: _event_ms(fn, reps, stream)
    out = {}

    # MP / AP / nearest-neighbour upsampling over SC(2, 2), 128^3 x 4 shapes, C = 64
    sc = sscn.sc_rulebook_build(tc, size, 2, 2)
    n_in, n_out, P = sc.n_in, sc.n_out, sc.n_pairs
    pool = {"workload": "sc2x2x2s2_grid128_shapes_c64", "n_in": n_in, "n_out": n_out, "pairs": P}
    for name, dt in (("f32", torch.float32), ("bf16", torch.bfloat16)):
        e = 4 if dt == torch.float32 else 2
        X = torch.from_numpy(S.features(n_in, 64, S.SEED_FEAT + 41)).to(dt).to(dev)
        G = torch.from_numpy(S.features(n_out, 64, S.SEED_GRAD + 41)).to(dt).to(dev)
        _, arg = sscn.pool_forward(X, sc, "max")
        xb, yb, ab, pb = n_in * 64 * e, n_out * 64 * e, n_out * 64, 8 * P
        pool[name] = {
            "max_forward": _hbm(xb + yb + ab + pb, timed(lambda: sscn.pool_forward(X, sc, "max"))),
            "max_backward": _hbm(yb + ab + xb + pb, timed(lambda: sscn.pool_backward(G, sc, "max", arg))),
            "avg_forward": _hbm(xb + yb + pb, timed(lambda: sscn.pool_forward(X, sc, "avg"))),
            "avg_backward": _hbm(yb + xb + pb, timed(lambda: sscn.pool_backward(G, sc, "avg"))),
            "upsample_forward": _hbm(yb + xb + pb, timed(lambda: sscn.upsample_forward(G, sc))),
            "upsample_backward": _hbm(xb + yb + pb, timed(lambda: sscn.upsample_backward(X, sc))),
        }
    out["pool"] = pool

    # batch normalisation over the active sites: the U-Net's level-0 size
    # (256^3 x 8 scenes, 32 channels, bf16) and the 64-channel layer (fp32)
    c256 = S.scenes_256()
    bn = {}
    for name, n, c, dt in (("scenes256_c32_bf16", int(c256.shape[0]), 32, torch.bfloat16),
                           ("shapes128_c64_f32", int(tc.shape[0]), 64, torch.float32)):
        e = 4 if dt == torch.float32 else 2
        x = (torch.from_numpy(S.features(n, c, S.SEED_FEAT + 42)) * 2 + 0.5).to(dt).to(dev)
        dA = torch.from_numpy(S.features(n, c, S.SEED_GRAD + 42)).to(dt).to(dev)
        g = torch.ones(c, device=dev)
        b = torch.zeros(c, device=dev)
        st = sscn.batchnorm_forward(x, g, b)
        dg, db = sscn.batchnorm_relu_backward_params(dA, x, st, b)
        dx = torch.empty_like(x)
        nb = n * c * e
        bn[name] = {
            "stats": _hbm(nb, timed(lambda: sscn.batchnorm_forward(x, g, b))),
            "apply_relu": _hbm(2 * nb, timed(lambda: sscn.batchnorm_relu_apply(x, st, b))),
            "backward_params": _hbm(2 * nb, timed(lambda: sscn.batchnorm_relu_backward_params(dA, x, st, b))),
            "backward_input": _hbm(3 * nb, timed(lambda: sscn.batchnorm_relu_backward_input(dA, x, g, b, st, dg, db,
                                                                                           dx))),
        }
    out["batchnorm"] = bn

    # one whole U-Net training step (forward, backward, SGD) on 256^3 x 8 scenes, bf16
    t256 = torch.from_numpy(c256).to(dev)
    ncls = 20
    geom = train.Geometry(t256, (256, 256, 256))
    Pm = train.Params(unet.CHANNELS, ncls, lambda nm, k, ci, co: S.train_params(nm, k, ci, co),
                      dtype=torch.bfloat16)
    x0 = torch.from_numpy(S.features(c256.shape[0], unet.CHANNELS[0], S.SEED_FEAT + 43, bf16=True)).to(
        torch.bfloat16).to(dev)
    lab = torch.from_numpy(S.labels(c256.shape[0], ncls, 44)).to(dev)
    step_ms = _wall_ms(lambda: train.train_step(x0, lab, geom, Pm), 3)
    fl = 3 * unet.flops(geom)  # forward, dgrad and wgrad of every convolution (the head aside)
    out["unet_train_step"] = {"workload": "unet5_grid256_batch8_scenes_c32to160_bf16_20classes",
                              "ms": step_ms, "sites_per_s": c256.shape[0] / (step_ms * 1e-3),
                              "conv_flops": fl, "effective_tflops": fl / (step_ms * 1e-3) / 1e12}
    del geom, Pm, x0, lab
    # the small three-level network the oracle's training step is timed on
    cs = S.scenes_small(batch=2, L=32, target_per_sample=3000)
    ts = torch.from_numpy(cs).to(dev)
    ch3, ncls3 = (8, 16, 24), 6
    geom3 = train.Geometry(ts, (32, 32, 32), levels=3)
    P3 = train.Params(ch3, ncls3, lambda nm, k, ci, co: S.train_params(nm, k, ci, co))
    xs = torch.from_numpy(S.features(cs.shape[0], ch3[0], S.SEED_FEAT + 31)).to(dev)
    ls = torch.from_numpy(S.labels(cs.shape[0], ncls3, 32)).to(dev)
    out["unet3_train_step_scenes32"] = {"workload": "unet3_grid32_batch2_scenes_c8to24_f32_6classes",
                                        "sites": int(cs.shape[0]),
                                        "ms": _wall_ms(lambda: train.train_step(xs, ls, geom3, P3), reps)}
    del geom3, P3

    # pre-activated residual block (two SSC(3) convolutions), 128^3 x 4 shapes, C = 64 fp32
    rb = sscn.ssc_rulebook_build(tc, size, 3)
    n = int(tc.shape[0])
    X = torch.from_numpy(S.features(n, 64, S.SEED_FEAT + 45)).to(dev)
    ps = [tuple(torch.from_numpy(a).to(dev) for a in S.layer_params(f"res{i}", 27, 64, 64, bf16=False))
          for i in range(2)]
    fwd_ms = timed(lambda: blocks.residual_block(X, rb, *ps))
    G = torch.from_numpy(S.features(n, 64, S.SEED_GRAD + 45)).to(dev)

    def train_block():
        y, cache = blocks.residual_block_train(X, rb, *ps)
        blocks.residual_block_train_backward(G, cache)

    train_ms = _wall_ms(train_block, reps)
    fl2 = 2 * 2.0 * 64 * 64 * rb.n_pairs
    out["residual_block"] = {"workload": "ssc3x3x3_x2_grid128_shapes_c64_f32", "forward_ms": fwd_ms,
                             "forward_tflops": fl2 / (fwd_ms * 1e-3) / 1e12, "train_fwd_bwd_ms": train_ms,
                             "train_tflops": 3 * fl2 / (train_ms * 1e-3) / 1e12}
    # a layer with a bias and a residual added in its write-out
    W = ps[0][2]
    bias = torch.from_numpy(S.features(1, 64, 46)[0]).to(dev)
    plain_ms = timed(lambda: sscn.sparse_conv_forward(X, W, rb))
    ex_ms = timed(lambda: sscn.sparse_conv_forward_ex(X, W, rb, bias=bias, residual=X))
    out["bias_residual_layer"] = {"forward_ms": plain_ms, "forward_bias_residual_ms": ex_ms}

    # 4-d SSC(3) (81 offsets) on moving shells, 16 time steps of 48^3 x 2, C = 32 fp32
    c4 = S.moving_shells_4d()
    t4 = torch.from_numpy(c4).to(dev)
    size4 = (16, 48, 48, 48)
    build_ms = _wall_ms(lambda: sscn.ssc_rulebook_build(t4, size4, 3), reps)
    r4 = sscn.ssc_rulebook_build(t4, size4, 3)
    X4 = torch.from_numpy(S.features(c4.shape[0], 32, S.SEED_FEAT + 47)).to(dev)
    W4 = torch.from_numpy(S.weights(81, 32, 32, S.SEED_WEIGHT + 47)).to(dev)
    f4_ms = timed(lambda: sscn.sparse_conv_forward(X4, W4, r4))
    fl4 = 2.0 * 32 * 32 * r4.n_pairs
    out["layer_4d"] = {"workload": "ssc3x3x3x3_t16_grid48_batch2_shells_c32_f32", "sites": int(c4.shape[0]),
                       "pairs": int(r4.n_pairs), "rulebook_build_ms": build_ms, "forward_ms": f4_ms,
                       "forward_tflops": fl4 / (f4_ms * 1e-3) / 1e12}
    return out


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
    build_lat_ms = _latency_ms(lambda: sscn.ssc_rulebook_build(tc, size, 3), reps)

    timed = lambda fn: _event_ms(fn, reps, stream)
    fwd_ms = timed(lambda: sscn.sparse_conv_forward(tX, tW, rb))
    dgrad_ms = timed(lambda: sscn.sparse_conv_backward(None, tW, tG, rb, dgrad=True, wgrad=False))
    if args.copy_calibration:
        copy_calibration()
    wgrad_ms = timed(lambda: sscn.sparse_conv_backward(tX, tW, tG, rb, dgrad=False, wgrad=True))
    # the same wgrad with its work items' partial sums added in a fixed order
    sscn.set_deterministic(True)
    try:
        wgrad_det_ms = timed(lambda: sscn.sparse_conv_backward(tX, tW, tG, rb, dgrad=False, wgrad=True))
    finally:
        sscn.set_deterministic(False)
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
        "wgrad_deterministic_ms": wgrad_det_ms,
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
                                         "SSC 3^3 rule-book build incl. its row-block plan, 100k sites",
                                         pairs_ms=build_lat_ms),
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
        result["extra"] = {"sc_then_ssc": sc_then_ssc(tc, size, stream, reps),
                           "scaling_in_sites": scaling_in_sites(stream, reps), "unet": unet_scenes(stream, 5),
                           "ops": ops_extra(tc, size, stream, reps)}
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(coords, size, X, W, G, args.cpu_seconds)
        if not args.no_extra:
            result["cpu_baseline"]["ops"] = cpu_ops(coords, size)
    print(json.dumps(result))


if __name__ == "__main__":
    main()
