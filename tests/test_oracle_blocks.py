"""Pins of the oracle's bias term (Sec. 3 footnote) and pre-activated
residual blocks (Sec. 5) against dense torch: conv3d with a bias read at the
active outputs, and the block on a dense grid with masks (inference and
training form, gradients by autograd)."""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import sscn_oracle as O
from paper_1711_10275_amd import synthetic as S
from tests import dense_ref as R


def _set(seed, size, density=0.2):
    rng = np.random.default_rng(seed)
    occ = rng.random((2,) + tuple(size)) < density
    occ[:, 0, 0, 0] = True
    c = np.argwhere(occ).astype(np.int32)
    return c[rng.permutation(c.shape[0])]


@pytest.mark.parametrize("kind,f,s", [("ssc", 3, 1), ("sc", 2, 2), ("sc", 3, 2)])
def test_forward_bias_is_dense_conv3d_with_bias(kind, f, s):
    size = (8, 8, 8) if (f, s) == (2, 2) else (9, 9, 9)
    rng = np.random.default_rng(1)
    c = _set(2, size)
    X, W, b = rng.standard_normal((c.shape[0], 3)), rng.standard_normal((f ** 3, 3, 4)), rng.standard_normal(4)
    rb = O.ssc_rulebook(c, size, f) if kind == "ssc" else O.sc_rulebook(c, size, f, s)
    Bn = int(c[:, 0].max()) + 1
    y = F.conv3d(R.to_dense(c, X, size, Bn), R.torch_weight(W, f), bias=torch.from_numpy(b),
                 padding=(f - 1) // 2 if kind == "ssc" else 0, stride=s).numpy()
    oc = rb.out_coords.astype(np.int64)
    np.testing.assert_allclose(O.forward_bias(X, W, b, rb), y[oc[:, 0], :, oc[:, 1], oc[:, 2], oc[:, 3]],
                               rtol=1e-12, atol=1e-12)


def _block_params(rng, c, train):
    out = []
    for _ in range(2):
        g = rng.uniform(0.5, 1.5, c)
        b = rng.normal(0, 0.3, c)
        out.append((g, b, rng.standard_normal((27, c, c)) / np.sqrt(27 * c)))
    return out


def test_residual_block_inference_is_dense():
    size = (10, 10, 10)
    rng = np.random.default_rng(3)
    c = _set(4, size)
    X = rng.standard_normal((c.shape[0], 6))
    p1, p2 = _block_params(rng, 6, False)
    rb = O.ssc_rulebook(c, size, 3)
    want, _ = R.dense_residual_block(c, size, X, p1, p2)
    np.testing.assert_allclose(O.residual_block(X, rb, p1, p2), want, rtol=1e-11, atol=1e-11)


def test_residual_block_training_matches_autograd():
    size = (10, 10, 10)
    rng = np.random.default_rng(5)
    c = _set(6, size)
    X = rng.standard_normal((c.shape[0], 5)) * 2 + 0.5
    p1, p2 = _block_params(rng, 5, True)
    rb = O.ssc_rulebook(c, size, 3)
    G = rng.standard_normal((c.shape[0], 5))
    Y, cache = O.residual_block_train(X, rb, p1, p2)
    want, grads = R.dense_residual_block(c, size, X, p1, p2, train=True, G=G)
    np.testing.assert_allclose(Y, want, rtol=1e-11, atol=1e-11)
    dX, g1, g2 = O.residual_block_train_backward(G, cache)
    np.testing.assert_allclose(dX, grads[0], rtol=1e-9, atol=1e-11)
    for got, ref in zip(g1 + g2, grads[1] + grads[2]):
        np.testing.assert_allclose(got, ref, rtol=1e-9, atol=1e-11)
