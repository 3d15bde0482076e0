"""Bias term and residual blocks on the GPU against the oracle."""
import numpy as np
import pytest
import torch

from oracle import sscn_oracle as O
from paper_1711_10275_amd import blocks, sscn
from paper_1711_10275_amd import synthetic as S
from tests.gpu_common import coords_for, dev, host, small_set
from tests.parity import assert_close, assert_close_head

pytestmark = pytest.mark.gpu

TD = {"f32": torch.float32, "bf16": torch.bfloat16}


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("kind,cin,cout", [("ssc", 64, 64), ("ssc", 16, 24), ("ssc", 12, 20), ("sc", 32, 48),
                                           ("dc", 48, 32)])
def test_forward_bias_and_residual(kind, cin, cout, dtype):
    """Bias alone, and bias + residual with an activated second head, over
    the row-block, generic and SC / DC paths."""
    size = (16, 16, 16)
    c = small_set(600 + cin, size, batch=2, density=0.2)
    bf = dtype == "bf16"
    if kind == "ssc":
        rb, orb = sscn.ssc_rulebook_build(dev(c), size, 3), O.ssc_rulebook(c, size, 3)
    else:
        rb, orb = sscn.sc_rulebook_build(dev(c), size, 2, 2), O.sc_rulebook(c, size, 2, 2)
        if kind == "dc":
            rb, orb = rb.transpose(), O.transpose(orb)
    X = S.features(orb.n_in, cin, 610 + cin, bf16=bf)
    W = S.weights(orb.K, cin, cout, 611 + cin, bf16=bf)
    rng = np.random.default_rng(cin)
    bias = rng.normal(0, 0.5, cout).astype(np.float32)
    res = S.features(orb.n_out, cout, 612 + cin, bf16=bf)
    y = sscn.sparse_conv_forward_ex(dev(X, TD[dtype]), dev(W, TD[dtype]), rb, bias=dev(bias))
    assert_close(host(y), O.forward_bias(X, W, bias, orb), dtype, "bias")
    scale = rng.uniform(0.5, 1.5, cout).astype(np.float32)
    shift = rng.normal(0, 0.1, cout).astype(np.float32)
    plain = torch.empty((orb.n_out, cout), dtype=TD[dtype], device="cuda:0")
    act = torch.empty((orb.n_out, cout), dtype=TD[dtype], device="cuda:0")
    sscn.sparse_conv_forward_heads(dev(X, TD[dtype]), dev(W, TD[dtype]), rb,
                                   [(plain, None, None), (act, dev(scale), dev(shift))],
                                   bias=dev(bias), residual=dev(res, TD[dtype]))
    ref = O.forward_bias(X, W, bias, orb) + res
    assert_close(host(plain), ref, dtype, "bias + residual")
    assert_close_head(host(act), ref, scale, shift, dtype, "activated head")


def _params(c, seed, bf16):
    out = []
    for i in range(2):
        s, t, w = S.layer_params(f"block{i}", 27, c, c, seed=seed, bf16=bf16)
        out.append((s, t, w))
    return out


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("config,c", [("shell32", 16), ("shapes128", 64)])
def test_residual_block_inference(config, c, dtype):
    coords, size = coords_for(config)
    bf = dtype == "bf16"
    rb, orb = sscn.ssc_rulebook_build(dev(coords), size, 3), O.ssc_rulebook(coords, size, 3)
    X = S.features(coords.shape[0], c, 620 + c, bf16=bf)
    p1, p2 = _params(c, 621, bf)
    tp = [(dev(s), dev(t), dev(w, TD[dtype])) for s, t, w in (p1, p2)]
    y = blocks.residual_block(dev(X, TD[dtype]), rb, *tp)
    # the oracle with the stored activations rounded as the GPU stores them
    rnd = O.round_bf16 if bf else (lambda a: a)
    a1 = rnd(O.affine_relu(X, p1[0], p1[1]))
    a2 = rnd(O.affine_relu(O.forward(a1, p1[2], orb), p2[0], p2[1]))
    assert_close(host(y), X + O.forward(a2, p2[2], orb), dtype, "residual block")


def test_residual_block_training_fp32():
    coords, size = coords_for("shapes128")
    c = 32
    rb, orb = sscn.ssc_rulebook_build(dev(coords), size, 3), O.ssc_rulebook(coords, size, 3)
    X = S.features(coords.shape[0], c, 630) * 2 + 0.5
    p1, p2 = _params(c, 631, False)
    G = S.features(coords.shape[0], c, 632)
    tp = [(dev(s), dev(t), dev(w)) for s, t, w in (p1, p2)]
    y, cache = blocks.residual_block_train(dev(X), rb, *tp)
    Y, ocache = O.residual_block_train(X, orb, p1, p2)
    assert_close(host(y), Y, "f32", "block output")
    dx, g1, g2 = blocks.residual_block_train_backward(dev(G), cache)
    rdx, r1, r2 = O.residual_block_train_backward(G, ocache)
    assert_close(host(dx), rdx, "f32", "dx")
    for got, want, what in zip(g1 + g2, r1 + r2, ["dgamma1", "dbeta1", "dW1", "dgamma2", "dbeta2", "dW2"]):
        assert_close(host(got), want, "f32", what)
