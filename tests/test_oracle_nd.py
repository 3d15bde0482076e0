"""Pins of the oracle in d = 1, 2 and 4 dimensions (Sec. 1: 4-D data such as
RGB-D video; Sec. 3 defines the layers for any d): dense conv1d / conv2d, a
4-D dense reference from conv3d slices, pure-Python brute-force triples,
and a 4-D grid with a single position along its last axis, which must give
the 3-D rule book."""
import numpy as np
import pytest

from oracle import sscn_oracle as O
from tests import dense_ref as R


def _set(seed, size, batch=2, density=0.3):
    rng = np.random.default_rng(seed)
    occ = rng.random((batch,) + tuple(size)) < density
    occ[(slice(None),) + (0,) * len(size)] = True
    occ[(slice(None),) + tuple(L - 1 for L in size)] = True
    c = np.argwhere(occ).astype(np.int32)
    return c[rng.permutation(c.shape[0])]


def brute_triples(coords, out_coords, f, s, submanifold):
    d = coords.shape[1] - 1
    c = (f - 1) // 2 if submanifold else 0
    step = 1 if submanifold else s
    out = []
    for j, (bj, *xj) in enumerate(coords.tolist()):
        for k, (bk, *yk) in enumerate(out_coords.tolist()):
            if bj != bk:
                continue
            i = [xj[q] - step * yk[q] + c for q in range(d)]
            if all(0 <= v < f for v in i):
                o = 0
                for v in i:
                    o = o * f + v
                out.append((j, k, o))
    return sorted(out, key=lambda t: (t[2], t[1], t[0]))


CASES = [((11,), 3, 1, True), ((12,), 2, 2, False), ((9, 7), 3, 1, True), ((9, 9), 3, 2, False),
         ((8, 6), 2, 2, False), ((6, 5, 4, 5), 3, 1, True), ((6, 6, 4, 4), 2, 2, False), ((5, 5, 5, 5), 3, 2, False)]


@pytest.mark.parametrize("size,f,s,sub", CASES)
def test_nd_rulebook_and_forward(size, f, s, sub):
    rng = np.random.default_rng(len(size) * 10 + f + s)
    c = _set(f + s + len(size), size, density=0.3 if len(size) < 4 else 0.15)
    rb = O.ssc_rulebook(c, size, f) if sub else O.sc_rulebook(c, size, f, s)
    assert rb.K == f ** len(size) and rb.d == len(size)
    assert O.canonical_triples(rb).tolist() == [list(t) for t in brute_triples(c, rb.out_coords, f, s, sub)]
    X, W = rng.standard_normal((c.shape[0], 3)), rng.standard_normal((rb.K, 3, 2))
    act, vals = R.dense_nd(c, X, W, size, f, s, sub)
    got = {tuple(r): i for i, r in enumerate(rb.out_coords.tolist())}
    assert sorted(got) == [tuple(r) for r in act.tolist()]
    Y = O.forward(X, W, rb)
    np.testing.assert_allclose(Y[[got[tuple(r)] for r in act.tolist()]], vals, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("f,s,sub", [(3, 1, True), (1, 1, True), (2, 2, False), (3, 2, False)])
def test_4d_with_one_position_on_the_last_axis_is_3d(f, s, sub):
    """A 4-D grid of extent 1 (SSC) or f (SC, so that one output position
    remains) along its last axis, every site at position 0 there: only
    offsets with last index = the centre (SSC) or 0 (SC) can connect, and
    they give the 3-D rule book of the first three axes."""
    size3 = (8, 8, 8) if (f, s) == (2, 2) else (9, 9, 9)
    c3 = _set(40 + f, size3, density=0.2)
    c4 = np.concatenate([c3, np.zeros((c3.shape[0], 1), np.int32)], axis=1)
    L3 = 1 if sub else f
    size4 = size3 + (L3,)
    rb3 = O.ssc_rulebook(c3, size3, f) if sub else O.sc_rulebook(c3, size3, f, s)
    rb4 = O.ssc_rulebook(c4, size4, f) if sub else O.sc_rulebook(c4, size4, f, s)
    keep = (f - 1) // 2 if sub else 0
    np.testing.assert_array_equal(rb4.out_coords[:, :4], rb3.out_coords)
    for o4 in range(rb4.K):
        o3, last = divmod(o4, f)
        if last == keep:
            np.testing.assert_array_equal(rb4.ins[o4], rb3.ins[o3])
            np.testing.assert_array_equal(rb4.outs[o4], rb3.outs[o3])
        else:
            assert rb4.ins[o4].size == 0


def test_nd_shape_errors():
    c = np.zeros((1, 3), np.int32)
    with pytest.raises(O.InvalidArg):
        O.ssc_rulebook(c, (4, 4, 4), 3)          # coords of a 2-D grid, 3 extents
    with pytest.raises(O.ShapeError):
        O.sc_rulebook(c, (5, 4), 2, 2)
