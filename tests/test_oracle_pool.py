"""Pins of the oracle's pooling and upsampling (Sec. 4.1 "Other operators":
MP takes the maximum of the zero vector and the active inputs of a field,
AP f^-d times their sum; Sec. 5: nearest-neighbour upsampling of the FCN)
against dense torch routines on grids where inactive sites hold zeros, and
their gradients against torch autograd."""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import sscn_oracle as O
from tests import dense_ref as R


def _set(seed, size, batch=2, density=0.25):
    rng = np.random.default_rng(seed)
    occ = rng.random((batch,) + tuple(size)) < density
    occ[:, 0, 0, 0] = True
    occ[:, -1, -1, -1] = True
    c = np.argwhere(occ).astype(np.int32)
    return c[rng.permutation(c.shape[0])]


def _at(y, coords):
    coords = np.asarray(coords, np.int64)
    return y[coords[:, 0], :, coords[:, 1], coords[:, 2], coords[:, 3]]


CASES = [((8, 8, 8), 2, 2), ((9, 9, 9), 3, 2), ((9, 9, 9), 3, 3), ((9, 9, 9), 1, 2)]


@pytest.mark.parametrize("size,f,s", CASES)
def test_max_pool_is_relu_of_dense_max_pool(size, f, s):
    rng = np.random.default_rng(11)
    c = _set(1, size)
    X = rng.standard_normal((c.shape[0], 5))
    rb = O.sc_rulebook(c, size, f, s)
    Y, A = O.max_pool(X, rb)
    B = int(c[:, 0].max()) + 1
    Xd = R.to_dense(c, X, size, B).requires_grad_(True)
    yd = torch.relu(F.max_pool3d(Xd, kernel_size=f, stride=s))
    np.testing.assert_array_equal(Y, _at(yd.detach().numpy(), rb.out_coords))
    # the field of an active output holds an active input; where all of its
    # inputs are negative the zero vector wins and no offset is recorded
    assert np.all((A == O.NO_ARGMAX) == (Y == 0.0))
    G = rng.standard_normal(Y.shape)
    oc = rb.out_coords.astype(np.int64)
    (yd[oc[:, 0], :, oc[:, 1], oc[:, 2], oc[:, 3]] * torch.from_numpy(G)).sum().backward()
    # (overlapping fields, f > s: an input's gradient sums over its outputs)
    np.testing.assert_allclose(O.max_pool_backward(G, A, rb), _at(Xd.grad.numpy(), c), rtol=1e-13, atol=1e-13)


def test_max_pool_ties_go_to_the_smallest_offset():
    """Equal maxima in one field: the input at the smallest offset o takes the
    gradient (pure-Python brute force over the field)."""
    size = (4, 4, 4)
    c = np.argwhere(np.ones((1,) + size, bool)).astype(np.int32)
    rng = np.random.default_rng(3)
    X = rng.integers(-2, 3, (c.shape[0], 3)).astype(np.float64)     # many ties
    rb = O.sc_rulebook(c, size, 2, 2)
    Y, A = O.max_pool(X, rb)
    row = {tuple(r): i for i, r in enumerate(c.tolist())}
    for k, (b, y0, y1, y2) in enumerate(rb.out_coords.tolist()):
        for ch in range(3):
            best, arg = 0.0, O.NO_ARGMAX
            for o in range(8):
                i = (o // 4, (o // 2) % 2, o % 2)
                v = X[row[(b, 2 * y0 + i[0], 2 * y1 + i[1], 2 * y2 + i[2])], ch]
                if v > best:
                    best, arg = v, o
            assert Y[k, ch] == best and A[k, ch] == arg


@pytest.mark.parametrize("size,f,s", CASES)
def test_avg_pool_is_dense_avg_pool(size, f, s):
    rng = np.random.default_rng(12)
    c = _set(2, size)
    X = rng.standard_normal((c.shape[0], 4))
    rb = O.sc_rulebook(c, size, f, s)
    B = int(c[:, 0].max()) + 1
    Xd = R.to_dense(c, X, size, B).requires_grad_(True)
    yd = F.avg_pool3d(Xd, kernel_size=f, stride=s)
    Y = O.avg_pool(X, rb)
    np.testing.assert_allclose(Y, _at(yd.detach().numpy(), rb.out_coords), rtol=1e-13, atol=1e-13)
    G = rng.standard_normal(Y.shape)
    oc = rb.out_coords.astype(np.int64)
    (yd[oc[:, 0], :, oc[:, 1], oc[:, 2], oc[:, 3]] * torch.from_numpy(G)).sum().backward()
    np.testing.assert_allclose(O.avg_pool_backward(G, rb), _at(Xd.grad.numpy(), c), rtol=1e-13, atol=1e-13)


@pytest.mark.parametrize("size,s", [((8, 8, 8), 2), ((9, 9, 9), 3), ((6, 8, 10), 2)])
def test_upsample_is_dense_nearest(size, s):
    rng = np.random.default_rng(13)
    c = _set(3, size)
    rb = O.sc_rulebook(c, size, s, s)
    Y = rng.standard_normal((rb.n_out, 3))
    B = int(c[:, 0].max()) + 1
    Yd = R.to_dense(rb.out_coords, Y, rb.out_size, B).requires_grad_(True)
    ud = F.interpolate(Yd, scale_factor=s, mode="nearest")
    assert tuple(ud.shape[2:]) == tuple(size)
    np.testing.assert_array_equal(O.upsample_nearest(Y, rb), _at(ud.detach().numpy(), c))
    G = rng.standard_normal((c.shape[0], 3))
    (ud[c[:, 0], :, c[:, 1], c[:, 2], c[:, 3]] * torch.from_numpy(G)).sum().backward()
    np.testing.assert_allclose(O.upsample_nearest_backward(G, rb), _at(Yd.grad.numpy(), rb.out_coords),
                               rtol=1e-13, atol=1e-13)


def test_pooling_argument_errors():
    c = _set(4, (8, 8, 8))
    with pytest.raises(O.InvalidArg):
        O.max_pool(np.zeros((c.shape[0], 2)), O.ssc_rulebook(c, (8, 8, 8), 3))
    with pytest.raises(O.InvalidArg):
        O.upsample_nearest(np.zeros((1, 2)), O.sc_rulebook(c, (9, 9, 9), 3, 2))
