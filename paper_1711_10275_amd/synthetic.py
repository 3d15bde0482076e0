"""Seeded synthetic inputs for the SSC / SC layers.

This module only *draws* inputs: voxelised surfaces (sphere shells, planar
patches, cylinder shells) standing in for the voxelised point clouds of the
paper's experiments (Sec. 6.1, 6.2: 2-3k-point ShapeNet objects, about 99%
empty voxels at S=48; Sec. 6.6: indoor scenes), plus Gaussian features,
weights and upstream gradients.  It holds none of the method's arithmetic: no
hashing, no rulebooks, no convolution.  Both the CPU oracle and the GPU path
read exactly the arrays produced here.

Coordinates are int32 ``n x 4`` rows ``(b, x0, x1, x2)`` sorted ascending and
de-duplicated.  bf16 inputs are the fp32 draws rounded to the nearest bf16
(ties to even) and returned as float32 arrays whose values are exactly
representable in bf16.
"""
from __future__ import annotations

import dataclasses
import zlib

import numpy as np

# Seed bases: geometry, features, weights, upstream gradient (+ config index).
SEED_GEOM, SEED_FEAT, SEED_WEIGHT, SEED_GRAD = 1000, 2000, 3000, 4000


# --------------------------------------------------------------------------
# voxelisers (float64, evaluated over each shape's bounding box)
# --------------------------------------------------------------------------
def _grid_box(lo, hi, L):
    lo = np.maximum(np.floor(lo).astype(np.int64), 0)
    hi = np.minimum(np.ceil(hi).astype(np.int64), L - 1)
    if np.any(hi < lo):
        return np.zeros((0, 3), np.int64)
    axes = [np.arange(lo[i], hi[i] + 1) for i in range(3)]
    g = np.stack(np.meshgrid(*axes, indexing="ij"), axis=-1)
    return g.reshape(-1, 3)


def sphere_shell(q, r, L):
    """Voxels p with | |p-q| - r | < 0.5."""
    q = np.asarray(q, np.float64)
    p = _grid_box(q - r - 1, q + r + 1, L)
    d = np.linalg.norm(p - q, axis=1)
    return p[np.abs(d - r) < 0.5]


def _orthonormal(nrm):
    nrm = nrm / np.linalg.norm(nrm)
    t = np.array([1.0, 0.0, 0.0]) if abs(nrm[0]) < 0.9 else np.array([0.0, 1.0, 0.0])
    u = np.cross(nrm, t)
    u /= np.linalg.norm(u)
    v = np.cross(nrm, u)
    return nrm, u, v


def plane_patch(q, nrm, w, h, L, rot=0.0):
    """Voxels p with |n.(p-q)| < 0.5, |u.(p-q)| <= w, |v.(p-q)| <= h."""
    q = np.asarray(q, np.float64)
    nrm, u, v = _orthonormal(np.asarray(nrm, np.float64))
    c, s = np.cos(rot), np.sin(rot)
    u, v = c * u + s * v, -s * u + c * v
    ext = np.abs(u) * w + np.abs(v) * h + 1.0
    # Walk the dominant axis of the normal analytically instead of testing the
    # whole bounding box (keeps large floors and walls cheap).
    ax = int(np.argmax(np.abs(nrm)))
    o1, o2 = [i for i in range(3) if i != ax]
    lo, hi = q - ext, q + ext
    a1 = np.arange(max(int(np.floor(lo[o1])), 0), min(int(np.ceil(hi[o1])), L - 1) + 1)
    a2 = np.arange(max(int(np.floor(lo[o2])), 0), min(int(np.ceil(hi[o2])), L - 1) + 1)
    if a1.size == 0 or a2.size == 0:
        return np.zeros((0, 3), np.int64)
    g1, g2 = np.meshgrid(a1, a2, indexing="ij")
    g1, g2 = g1.ravel(), g2.ravel()
    # n.(p-q) = 0 solved for the dominant coordinate, then +-1 voxel around it
    rest = nrm[o1] * (g1 - q[o1]) + nrm[o2] * (g2 - q[o2])
    xc = q[ax] - rest / nrm[ax]
    pts = []
    for dz in (-1, 0, 1):
        xa = np.round(xc).astype(np.int64) + dz
        p = np.zeros((g1.size, 3), np.int64)
        p[:, ax], p[:, o1], p[:, o2] = xa, g1, g2
        pts.append(p)
    p = np.concatenate(pts)
    p = p[(p[:, ax] >= 0) & (p[:, ax] < L)]
    dp = p - q
    keep = (np.abs(dp @ nrm) < 0.5) & (np.abs(dp @ u) <= w) & (np.abs(dp @ v) <= h)
    return p[keep]


def cylinder_shell(q, axis, r, h, L):
    """Voxels p with | |(p-q) - ((p-q).a)a| - r | < 0.5 and |(p-q).a| <= h."""
    q = np.asarray(q, np.float64)
    a = np.asarray(axis, np.float64)
    a = a / np.linalg.norm(a)
    ext = r + h + 1
    p = _grid_box(q - ext, q + ext, L)
    dp = p - q
    t = dp @ a
    radial = np.linalg.norm(dp - t[:, None] * a[None, :], axis=1)
    return p[(np.abs(radial - r) < 0.5) & (np.abs(t) <= h)]


def _unit(rng):
    v = rng.normal(size=3)
    return v / np.linalg.norm(v)


def _random_object(rng, L, scale):
    kind = rng.integers(0, 3)
    q = rng.uniform(0.3 * L, 0.7 * L, size=3)
    if kind == 0:
        return sphere_shell(q, rng.uniform(10, 22) * scale, L)
    if kind == 1:
        return plane_patch(q, _unit(rng), rng.uniform(12, 24) * scale,
                           rng.uniform(12, 24) * scale, L, rot=rng.uniform(0, np.pi))
    return cylinder_shell(q, _unit(rng), rng.uniform(6, 14) * scale,
                          rng.uniform(12, 24) * scale, L)


def _finish(per_sample):
    """Stack (b, p) rows, de-duplicate, sort ascending by (b, x0, x1, x2)."""
    rows = []
    for b, p in enumerate(per_sample):
        if p.shape[0] == 0:
            continue
        rows.append(np.concatenate([np.full((p.shape[0], 1), b, np.int64), p], axis=1))
    if not rows:
        return np.zeros((0, 4), np.int32)
    c = np.unique(np.concatenate(rows), axis=0)  # np.unique sorts rows lexicographically
    return c.astype(np.int32)


# --------------------------------------------------------------------------
# workloads
# --------------------------------------------------------------------------
def shell_32(seed=SEED_GEOM + 0):
    """One sphere shell, radius 12, centre 16 + U(-1,1)^3, in a 32^3 grid."""
    rng = np.random.default_rng(seed)
    q = 16.0 + rng.uniform(-1, 1, size=3)
    return _finish([sphere_shell(q, 12.0, 32)])


def shapes_128(seed=SEED_GEOM + 1, batch=4, shapes=8, L=128, target=100_000):
    """Batch of samples, each the union of `shapes` random surfaces.

    The size ranges are scaled by one common factor, chosen by a short
    deterministic search, so that the whole batch lands within 10% of
    `target` active sites.
    """
    scale = 1.0
    for _ in range(12):
        rng = np.random.default_rng(seed)
        per = []
        for _b in range(batch):
            parts = [_random_object(rng, L, scale) for _ in range(shapes)]
            per.append(np.concatenate(parts) if parts else np.zeros((0, 3), np.int64))
        c = _finish(per)
        n = c.shape[0]
        if target is None or abs(n - target) <= 0.1 * target:
            return c
        scale *= np.sqrt(target / max(n, 1))  # surface area ~ scale^2
    return c


def scenes_256(seed=SEED_GEOM + 3, batch=8, L=256, target_per_sample=250_000):
    """Indoor-like scenes: floor, walls and at least 20 objects per sample.

    Floor and walls are large axis-aligned planar patches; objects are random
    sphere shells, cylinder shells and tilted patches.  Objects are added
    until the sample holds `target_per_sample` sites (within 10%); an object
    that would overshoot by more than 8% is redrawn.  Object sizes scale
    with L / 256.
    """
    g = L / 256.0
    per = []
    for b in range(batch):
        rng = np.random.default_rng(seed * 1000 + b)
        occ = np.zeros((L, L, L), bool)
        h = L / 2 - 1
        for p in (plane_patch([L / 2, L / 2, 8.0], [0, 0, 1], h, h, L),          # floor
                  plane_patch([8.0, L / 2, L / 2], [1, 0, 0], h, h / 2, L),      # walls
                  plane_patch([L - 9.0, L / 2, L / 2], [1, 0, 0], h, h / 2, L),
                  plane_patch([L / 2, 8.0, L / 2], [0, 1, 0], h, h / 2, L)):
            occ[p[:, 0], p[:, 1], p[:, 2]] = True
        count = int(occ.sum())
        n_obj = 0
        for _ in range(2000):
            if count >= 0.97 * target_per_sample and n_obj >= 20:
                break
            q = np.array([rng.uniform(16 * g, L - 16 * g), rng.uniform(16 * g, L - 16 * g),
                          rng.uniform(12 * g, L / 2)])
            kind = rng.integers(0, 3)
            s = rng.uniform(1.0, 1.8)
            if kind == 0:
                obj = sphere_shell(q, rng.uniform(8, 22) * s * g, L)
            elif kind == 1:
                obj = plane_patch(q, _unit(rng), rng.uniform(10, 24) * s * g, rng.uniform(10, 24) * s * g, L,
                                  rot=rng.uniform(0, np.pi))
            else:
                obj = cylinder_shell(q, _unit(rng), rng.uniform(5, 14) * s * g, rng.uniform(10, 24) * s * g, L)
            new = int(np.count_nonzero(~occ[obj[:, 0], obj[:, 1], obj[:, 2]]))
            if count + new > 1.08 * target_per_sample:
                continue
            occ[obj[:, 0], obj[:, 1], obj[:, 2]] = True
            count = int(occ.sum())
            n_obj += 1
        per.append(np.argwhere(occ))
    return _finish(per)


# --------------------------------------------------------------------------
# dense draws
# --------------------------------------------------------------------------
def bf16_round(a):
    """Round float32 values to the nearest bfloat16 (ties to even); float32 out."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    r = ((u + 0x7FFF + lsb) >> 16) << 16
    nan = np.isnan(a)
    out = (r & 0xFFFFFFFF).astype(np.uint32).view(np.float32).copy()
    out[nan] = np.nan
    return out


def shuffled(coords, seed):
    """The same active sites with their rows in a seeded random order (the
    locality-sensitivity run: feature rows no longer follow the grid)."""
    return np.ascontiguousarray(coords[np.random.default_rng(seed).permutation(coords.shape[0])])


def features(n, c, seed, bf16=False):
    x = np.random.default_rng(seed).standard_normal((n, c), dtype=np.float32)
    return bf16_round(x) if bf16 else x


def weights(k, cin, cout, seed, bf16=False):
    """W[o][ci][co] ~ N(0, 1/(k*cin))."""
    w = np.random.default_rng(seed).standard_normal((k, cin, cout), dtype=np.float32)
    w *= np.float32(1.0 / np.sqrt(k * cin))
    return bf16_round(w) if bf16 else w


def layer_params(name, k, cin, cout, seed=SEED_WEIGHT + 3, bf16=True):
    """Parameters of one named network layer: a per-input-channel affine map
    (inference-form batch normalisation: scale ~ U(0.5, 1.5), shift ~
    N(0, 0.1)) and weights W[o][ci][co] ~ N(0, 1/(k cin)).

    The draw depends only on (seed, name, k, cin, cout), so any code that
    names its layers the same way gets the same parameters.
    """
    s = seed * 1_000_003 + zlib.crc32(name.encode()) + 7919 * (k * 1_000_000 + cin * 1000 + cout)
    rng = np.random.default_rng(s)
    scale = rng.uniform(0.5, 1.5, cin).astype(np.float32)
    shift = rng.normal(0.0, 0.1, cin).astype(np.float32)
    return scale, shift, weights(k, cin, cout, s + 1, bf16=bf16)


def train_params(name, k, cin, cout, seed=SEED_WEIGHT + 5, bf16=False):
    """Parameters of one network layer for training: batch-normalisation
    gain ~ U(0.5, 1.5) and bias ~ N(0, 0.1) over the input channels, weights
    W[o][ci][co] ~ N(0, 1/(k cin)); the layer named "head" also gets a bias
    over its output channels ~ N(0, 0.1)."""
    scale, shift, w = layer_params(name, k, cin, cout, seed=seed, bf16=bf16)
    if name != "head":
        return scale, shift, w
    s = seed * 1_000_003 + zlib.crc32(name.encode()) + 17
    return scale, shift, w, np.random.default_rng(s).normal(0.0, 0.1, cout).astype(np.float32)


def labels(n, n_classes, seed):
    """One class per active site, uniform."""
    return np.random.default_rng(seed).integers(0, n_classes, n).astype(np.int32)


def moving_shells_4d(seed=SEED_GEOM + 21, batch=2, T=16, L=48, shells=3):
    """Sparse 4-d sets (time x a 3-d grid, the kind of data RGB-D video
    gives): per sample, sphere shells of radius U(8, 14) whose centres move
    linearly in time (up to L / 4 over the T steps), each time step
    voxelised like sphere_shell.  Rows (b, t, x0, x1, x2), sorted."""
    rng = np.random.default_rng(seed)
    rows = []
    for b in range(batch):
        objs = [(rng.uniform(0.35 * L, 0.65 * L, 3), rng.uniform(-0.25, 0.25, 3) * L / max(T - 1, 1),
                 rng.uniform(8, 14)) for _ in range(shells)]
        for t in range(T):
            pts = np.concatenate([sphere_shell(q + v * t, r, L) for q, v, r in objs])
            pts = np.unique(pts, axis=0)
            rows.append(np.concatenate([np.full((pts.shape[0], 1), b, np.int64), np.full((pts.shape[0], 1), t,
                                                                                      np.int64), pts], axis=1))
    c = np.unique(np.concatenate(rows), axis=0)
    return c.astype(np.int32)


def scenes_small(seed=SEED_GEOM + 13, batch=2, L=64, target_per_sample=15_000):
    """The indoor-scene recipe on a small grid (end-to-end network checks)."""
    return scenes_256(seed=seed, batch=batch, L=L, target_per_sample=target_per_sample)


@dataclasses.dataclass
class LayerInput:
    coords: np.ndarray          # int32 n x 4
    spatial_size: tuple         # (L0, L1, L2)
    features: np.ndarray        # float32 n x Cin (bf16-representable if bf16)
    weights: np.ndarray         # float32 K x Cin x Cout
    grad: np.ndarray | None     # float32 n_out x Cout, or None


def random_small(seed, L=8, batch=2, density=0.15, boundary=True):
    """Random active set on a tiny grid (for brute-force checks), sorted rows."""
    rng = np.random.default_rng(seed)
    occ = rng.random((batch, L, L, L)) < density
    if boundary:
        occ[:, 0, 0, 0] = True
        occ[:, L - 1, L - 1, L - 1] = True
    b, x0, x1, x2 = np.nonzero(occ)
    return np.stack([b, x0, x1, x2], axis=1).astype(np.int32)
