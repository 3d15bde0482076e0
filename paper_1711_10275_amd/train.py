"""One training step of the submanifold U-Net composed from the library's calls.

Network: the U-Net of unet.py (Sec. 5: pre-activated SSC(3) units, SC(2, 2)
down, DC(2, 2) up, skip concatenation), with every unit's batch
normalisation in training form -- statistics of its input over the active
sites (Sec. 4.1) -- followed by a head on the level-0 sites: batch
normalisation + ReLU and a per-site linear layer with bias (an SSC
convolution with filter size 1), softmax and the mean negative
log-likelihood of one label per site.  The step then updates every
parameter by SGD with Nesterov momentum and L2 weight decay (Sec. 6.2:
momentum 0.9, weight decay 1e-4, learning rate 0.1).

Every arithmetic step runs in libsscn.so; this module orders the calls and
keeps the tensors the backward pass needs (each unit's input and its
pre-activated input, and the batch statistics).  Parameters are kept in
fp32 (the master copy the update works on); a bf16 network convolves with a
bf16 copy of its weights, which the update refreshes.
"""
from __future__ import annotations

import torch

from . import sscn, unet


class Geometry(unet.Geometry):
    """unet.Geometry plus the filter-size-1 rule book of the level-0 sites (the head)."""

    def __init__(self, coords, spatial_size, levels=len(unet.CHANNELS)):
        super().__init__(coords, spatial_size, levels)
        self.head = sscn.ssc_rulebook_build(coords, spatial_size, 1)


class Params:
    """fp32 parameters, momentum buffers and running statistics of every
    unit ((gamma, beta, W) each) and of the head ((gamma, beta, W, bias),
    W of shape (1, C_0, n_classes)); `compute[name]` is W in the network's
    dtype."""

    def __init__(self, channels, n_classes, draw, dtype=torch.float32, device="cuda:0"):
        self.channels, self.n_classes, self.dtype = tuple(channels), n_classes, dtype
        self.master, self.buf, self.compute, self.running = {}, {}, {}, {}
        shapes = [(u.name, u.k, u.cin, u.cout) for u in unet.units(channels)]
        shapes.append(("head", 1, channels[0], n_classes))
        for name, k, cin, cout in shapes:
            vals = draw(name, k, cin, cout)
            ts = [torch.from_numpy(v).to(torch.float32).to(device).contiguous() for v in vals]
            self.master[name] = ts
            self.buf[name] = [torch.zeros_like(t) for t in ts]
            self.compute[name] = ts[2] if dtype == torch.float32 else ts[2].to(dtype)
            self.running[name] = (torch.zeros(cin, dtype=torch.float32, device=device),
                                  torch.ones(cin, dtype=torch.float32, device=device))

    def names(self):
        return list(self.master)


def _bn_relu(name, x, P, tape_entry):
    gamma, beta = P.master[name][0], P.master[name][1]
    rm, rv = P.running[name]
    st = sscn.batchnorm_forward(x, gamma, beta, running_mean=rm, running_var=rv)
    a = sscn.batchnorm_relu_apply(x, st, beta)
    tape_entry.update(x=x, a=a, st=st)
    return a


def _bn_relu_back(name, da, e, P, outs):
    """outs: [(tensor, (lo, hi), add or None)] column ranges of the gradient at e["x"]."""
    gamma, beta = P.master[name][0], P.master[name][1]
    dg, db = sscn.batchnorm_relu_backward_params(da, e["x"], e["st"], beta)
    for out, cols, add in outs:
        sscn.batchnorm_relu_backward_input(da, e["x"], gamma, beta, e["st"], dg, db, out, add=add, cols=cols)
    return dg, db


def train_step(x, labels, geom, P, lr=0.1, momentum=0.9, weight_decay=1e-4, update=True, trace=None):
    """Forward, backward and (if `update`) the SGD step on level-0 features
    x (n_0 x C_0, the network's dtype) and int32 labels (n_0).  Returns
    (loss (device fp32 scalar), grads {name: [dgamma, dbeta, dW(, dbias)]},
    fp32).  If `trace` is a dict it receives, per unit name, the tensors of
    that unit: x, a (its pre-activated input), y (its output), dy, da, dx."""
    channels = P.channels
    L = len(channels)
    if geom.levels != L:
        raise ValueError("channel list and geometry disagree on the number of levels")
    tape = []

    def unit(u, inp):
        e = {"u": u}
        a = _bn_relu(u.name, inp, P, e)
        y = sscn.sparse_conv_forward(a, P.compute[u.name], geom.rulebook(u))
        e["y"] = y
        tape.append(e)
        return y

    by_name = {u.name: u for u in unet.units(channels)}
    h, skips = x, {}
    for l in range(L):
        h = unit(by_name[f"enc{l}a"], h)
        h = unit(by_name[f"enc{l}b"], h)
        skips[l] = h
        if l < L - 1:
            h = unit(by_name[f"down{l}"], h)
    for l in reversed(range(L - 1)):
        up = unit(by_name[f"up{l}"], h)
        h = sscn.concat_cols(skips[l], up)
        h = unit(by_name[f"dec{l}a"], h)
        h = unit(by_name[f"dec{l}b"], h)
    head = {}
    z = _bn_relu("head", h, P, head)
    logits = sscn.sparse_conv_forward_ex(z, P.compute["head"], geom.head, bias=P.master["head"][3])
    loss, dlogits = sscn.softmax_nll(logits, labels)

    grads = {}
    dz, dWh = sscn.sparse_conv_backward(z, P.compute["head"], dlogits, geom.head)
    dbias = sscn.column_sum(dlogits)
    dx = torch.empty_like(h)
    dg, db = _bn_relu_back("head", dz, head, P, [(dx, None, None)])
    grads["head"] = [dg, db, dWh, dbias]
    if trace is not None:
        trace["head"] = dict(head, dy=dlogits, da=dz, dx=dx, logits=logits)

    def unit_back(dy, split=None, add=None):
        e = tape.pop()
        u = e["u"]
        da, dW = sscn.sparse_conv_backward(e["a"], P.compute[u.name], dy, geom.rulebook(u))
        if split is None:
            out = torch.empty_like(e["x"])
            outs, res = [(out, None, add)], out
        else:
            res = [torch.empty((e["x"].shape[0], hi - lo), dtype=e["x"].dtype, device=e["x"].device)
                   for lo, hi in split]
            outs = [(r, cols, None) for r, cols in zip(res, split)]
        dg, db = _bn_relu_back(u.name, da, e, P, outs)
        grads[u.name] = [dg, db, dW]
        if trace is not None:
            trace[u.name] = dict(e, dy=dy, da=da, dx=res)
        return res

    dskip = {}
    for l in range(L - 1):
        c = channels[l]
        dx = unit_back(dx)                                     # dec{l}b
        dskip[l], dup = unit_back(dx, split=[(0, c), (c, 2 * c)])  # dec{l}a: [skip | up] halves
        dx = unit_back(dup)                                    # up{l}: gradient at level l + 1
    for l in reversed(range(L)):
        if l < L - 1:
            dx = unit_back(dx, add=dskip.pop(l))               # down{l}, plus the skip's gradient
        dx = unit_back(dx)                                     # enc{l}b
        dx = unit_back(dx)                                     # enc{l}a
    assert not tape

    if update:
        for name, ts in P.master.items():
            for i, (p, g, b) in enumerate(zip(ts, grads[name], P.buf[name])):
                copy = P.compute[name] if (i == 2 and P.dtype != torch.float32) else None
                sscn.sgd_nesterov_(p, g.reshape(p.shape), b, lr, momentum, weight_decay, params_bf16=copy)
    return loss, grads
