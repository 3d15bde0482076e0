"""Rule-book build workload for the profiler.

Builds the SSC 3^3 rule book of the 256^3 x 8 scene set (about 2M active
sites, the first level of the U-Net) and the SC(2, 2) rule book from it,
`--reps` times each, then runs the measure library's 256 MiB copy (the
calibration of the FETCH_SIZE / WRITE_SIZE counters).  Prints one JSON line
with the sizes and the mean wall time of each build.  Measurement
infrastructure, not part of the layer path.

    python -u -m paper_1711_10275_amd.measure.builds [--reps N]
"""
from __future__ import annotations

import argparse
import ctypes
import json
import os
import time


def main():
    p = argparse.ArgumentParser()
    p.add_argument("--reps", type=int, default=3)
    args = p.parse_args()
    import torch
    from paper_1711_10275_amd import sscn
    from paper_1711_10275_amd import synthetic as S

    dev = torch.device("cuda:0")
    c = S.scenes_256()
    tc = torch.from_numpy(c).to(dev)
    size = (256, 256, 256)
    out = {"workload": "scenes256_batch8", "sites": int(c.shape[0])}

    def wall(fn):
        fn()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(args.reps):
            r = fn()
        torch.cuda.synchronize()
        return r, (time.perf_counter() - t0) * 1e3 / args.reps

    rb, out["ssc_build_ms"] = wall(lambda: sscn.ssc_rulebook_build(tc, size, 3))
    out["ssc_pairs"] = int(rb.n_pairs)
    del rb
    sc, out["sc_build_ms"] = wall(lambda: sscn.sc_rulebook_build(tc, size, 2, 2))
    out["sc_out_sites"], out["sc_pairs"] = int(sc.n_out), int(sc.n_pairs)
    del sc
    lib = ctypes.CDLL(os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                                   "libsscn_measure.so"))
    lib.sscn_measure_copy.argtypes = [ctypes.c_int64, ctypes.c_int, ctypes.POINTER(ctypes.c_double)]
    v = ctypes.c_double()
    lib.sscn_measure_copy(256 << 20, 2, ctypes.byref(v))
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
