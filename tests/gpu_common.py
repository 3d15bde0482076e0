"""Shared helpers for the GPU parity tests (inputs, oracle caching, transfers)."""
import functools

import numpy as np
import pytest
import torch

from paper_1711_10275_amd import synthetic as S


def device():
    if not torch.cuda.is_available():
        pytest.fail("GPU test selected but no GPU is visible")
    return torch.device("cuda:0")


def dev(a, dtype=None):
    """numpy -> device tensor; float arrays become float32 or bfloat16."""
    t = torch.from_numpy(np.ascontiguousarray(a))
    if dtype is not None:
        t = t.to(dtype)
    return t.to(device())


def host(t):
    return t.detach().float().cpu().numpy() if t.is_floating_point() else t.cpu().numpy()


@functools.lru_cache(maxsize=None)
def coords_for(config):
    """Active sites of the named workloads (cached per process)."""
    if config == "shell32":
        return S.shell_32(), (32, 32, 32)
    if config == "shapes128":
        return S.shapes_128(), (128, 128, 128)
    if config == "scenes256":
        return S.scenes_256(), (256, 256, 256)
    raise KeyError(config)


def small_set(seed, size, batch=2, density=0.15):
    rng = np.random.default_rng(seed)
    occ = rng.random((batch,) + tuple(size)) < density
    occ[:, 0, 0, 0] = True
    occ[:, -1, -1, -1] = True
    b, x0, x1, x2 = np.nonzero(occ)
    c = np.stack([b, x0, x1, x2], axis=1)
    return c[rng.permutation(c.shape[0])].astype(np.int32)


def gpu_offset_pairs(rb):
    """Per offset, (in, out) int64 arrays from the GPU export (sorted by out, in)."""
    i, o, off = (host(x).astype(np.int64) for x in rb.export())
    assert np.all(np.diff(off) >= 0), "export must be sorted by offset"
    res = []
    for q in range(rb.n_offsets):
        lo, hi = np.searchsorted(off, q), np.searchsorted(off, q, side="right")
        res.append((i[lo:hi], o[lo:hi]))
    return res


def oracle_offset_pairs(orb):
    res = []
    for q in range(orb.K):
        ins, outs = orb.ins[q], orb.outs[q]
        order = np.lexsort((ins, outs))
        res.append((ins[order].astype(np.int64), outs[order].astype(np.int64)))
    return res


def assert_same_rulebook(rb, orb, what=""):
    assert rb.n_in == orb.n_in and rb.n_out == orb.n_out, (what, rb.n_in, orb.n_in, rb.n_out, orb.n_out)
    assert rb.n_pairs == orb.n_pairs(), (what, rb.n_pairs, orb.n_pairs())
    assert rb.pairs_per_offset == orb.pairs_per_offset().tolist(), what
    g, o = gpu_offset_pairs(rb), oracle_offset_pairs(orb)
    for q in range(orb.K):
        np.testing.assert_array_equal(g[q][0], o[q][0], err_msg=f"{what} in rows, offset {q}")
        np.testing.assert_array_equal(g[q][1], o[q][1], err_msg=f"{what} out rows, offset {q}")


@functools.lru_cache(maxsize=None)
def oracle_levels(config, depth):
    """Oracle geometry of a U-Net: per level (coords, size, SSC(3) rule book,
    SC(2, 2) rule book or None), built from the level-0 sites of `config`."""
    from oracle import sscn_oracle as O
    coords, size = coords_for(config) if config != "scenes_small" else (S.scenes_small(), (64, 64, 64))
    out = []
    for l in range(depth):
        ssc = O.ssc_rulebook(coords, size, 3)
        sc = O.sc_rulebook(coords, size, 2, 2) if l + 1 < depth else None
        out.append((coords, size, ssc, sc))
        if sc is not None:
            coords, size = sc.out_coords, sc.out_size
    return tuple(out)
