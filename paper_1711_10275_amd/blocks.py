"""Pre-activated residual blocks (Sec. 5) composed from the library's calls.

A block holds two pre-activated SSC(3) units and an identity shortcut (the
numbers of input and output features are equal):

    y = x + SSC(relu(bn2(SSC(relu(bn1(x)), W1))), W2)

Inference form: bn is the per-channel affine map (scale, shift); the first
convolution writes its output already pre-activated for the second (an
output head), and the second adds the shortcut in its write-out, so each
intermediate is written once.  Training form: bn uses the batch statistics
of its input over the active sites (Sec. 4.1); the backward pass sends the
output gradient both through the units and, unchanged, along the shortcut.
Every arithmetic step runs in libsscn.so.
"""
from __future__ import annotations

import torch

from . import sscn


def residual_block(x, rb, p1, p2):
    """Inference form; p = (scale, shift, W) per unit (scale, shift fp32 over
    the unit's input channels, W [27][C][C] in x's dtype); rb: the level's
    SSC(3) rule book."""
    s1, t1, W1 = p1
    s2, t2, W2 = p2
    a1 = sscn.affine_relu(x, s1, t1)
    a2 = torch.empty_like(x)
    sscn.sparse_conv_forward_heads(a1, W1, rb, [(a2, s2, t2)])
    return sscn.sparse_conv_forward_ex(a2, W2, rb, residual=x)


def residual_block_train(x, rb, p1, p2):
    """Training form; p = (gamma, beta, W) per unit (gamma, beta fp32).
    Returns (y, cache for residual_block_train_backward)."""
    g1, b1, W1 = p1
    g2, b2, W2 = p2
    st1 = sscn.batchnorm_forward(x, g1, b1)
    a1 = sscn.batchnorm_relu_apply(x, st1, b1)
    h = sscn.sparse_conv_forward(a1, W1, rb)
    st2 = sscn.batchnorm_forward(h, g2, b2)
    a2 = sscn.batchnorm_relu_apply(h, st2, b2)
    y = sscn.sparse_conv_forward_ex(a2, W2, rb, residual=x)
    return y, (x, rb, p1, p2, st1, a1, h, st2, a2)


def residual_block_train_backward(dy, cache):
    """(dx, (dgamma1, dbeta1, dW1), (dgamma2, dbeta2, dW2)); dW fp32."""
    x, rb, (g1, b1, W1), (g2, b2, W2), st1, a1, h, st2, a2 = cache
    da2, dW2 = sscn.sparse_conv_backward(a2, W2, dy, rb)
    dg2, db2 = sscn.batchnorm_relu_backward_params(da2, h, st2, b2)
    dh = sscn.batchnorm_relu_backward_input(da2, h, g2, b2, st2, dg2, db2, torch.empty_like(h))
    da1, dW1 = sscn.sparse_conv_backward(a1, W1, dh, rb)
    dg1, db1 = sscn.batchnorm_relu_backward_params(da1, x, st1, b1)
    dx = sscn.batchnorm_relu_backward_input(da1, x, g1, b1, st1, dg1, db1, torch.empty_like(x), add=dy)
    return dx, (dg1, db1, dW1), (dg2, db2, dW2)
