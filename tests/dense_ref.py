"""Dense brute-force references used to pin the CPU oracle on tiny grids.

The sparse layers are dense convolutions restricted to active sites
(Sec. 4.1: inactive inputs read as zero; SSC outputs only at active input
sites; SC outputs where the receptive field holds an active input).  These
helpers scatter the sparse inputs into a dense zero grid, call torch's CPU
conv3d / conv_transpose3d in float64 (a library routine, cross-correlation),
and read the result back at the active output sites.  A second, pure numpy
loop implementation covers the SSC case without torch.
"""
import numpy as np
import torch
import torch.nn.functional as F


def to_dense(coords, X, size, batch=None):
    coords = np.asarray(coords, np.int64)
    X = np.asarray(X, np.float64)
    B = int(coords[:, 0].max()) + 1 if batch is None else batch
    C = X.shape[1]
    d = np.zeros((B, C) + tuple(size), np.float64)
    if coords.shape[0]:
        d[coords[:, 0], :, coords[:, 1], coords[:, 2], coords[:, 3]] = X
    return torch.from_numpy(d)


def torch_weight(W, f):
    """W[o][ci][co] (o = i0 f^2 + i1 f + i2) -> conv3d weight [co][ci][i0][i1][i2]."""
    W = np.asarray(W, np.float64)
    K, cin, cout = W.shape
    w = W.reshape(f, f, f, cin, cout).transpose(4, 3, 0, 1, 2)
    return torch.from_numpy(np.ascontiguousarray(w))


def dense_ssc(coords, X, W, size, f):
    """SSC via dense conv3d with padding (f-1)/2, read at the input sites."""
    coords = np.asarray(coords, np.int64)
    B = int(coords[:, 0].max()) + 1
    y = F.conv3d(to_dense(coords, X, size, B), torch_weight(W, f), padding=(f - 1) // 2)
    y = y.numpy()
    return y[coords[:, 0], :, coords[:, 1], coords[:, 2], coords[:, 3]]


def dense_sc(coords, X, W, size, f, s):
    """SC via dense conv3d with stride s.

    Returns (active output coords sorted by (b, y), features at them).  The
    active set is where conv3d of the occupancy with an all-ones filter is
    positive, i.e. the field holds at least one active input.
    """
    coords = np.asarray(coords, np.int64)
    B = int(coords[:, 0].max()) + 1
    occ = to_dense(coords, np.ones((coords.shape[0], 1)), size, B)
    cnt = F.conv3d(occ, torch.ones(1, 1, f, f, f, dtype=torch.float64), stride=s).numpy()[:, 0]
    act = np.argwhere(cnt > 0)
    y = F.conv3d(to_dense(coords, X, size, B), torch_weight(W, f), stride=s).numpy()
    vals = y[act[:, 0], :, act[:, 1], act[:, 2], act[:, 3]]
    return act.astype(np.int64), vals, cnt


def dense_dc(out_coords, Xdc, Wdc, in_coords, size, f, s):
    """DC (inverse of SC(f, s)) via conv_transpose3d, read at the SC input sites.

    Wdc[o][ci][co] maps the SC output features (ci) back to the SC input
    sites (co).  conv_transpose3d weight layout is [in][out][i0][i1][i2].
    """
    out_coords = np.asarray(out_coords, np.int64)
    in_coords = np.asarray(in_coords, np.int64)
    B = int(in_coords[:, 0].max()) + 1
    osize = tuple((L - f + s) // s for L in size)
    Wdc = np.asarray(Wdc, np.float64)
    K, cin, cout = Wdc.shape
    w = torch.from_numpy(np.ascontiguousarray(Wdc.reshape(f, f, f, cin, cout).transpose(3, 4, 0, 1, 2)))
    y = F.conv_transpose3d(to_dense(out_coords, Xdc, osize, B), w, stride=s).numpy()
    return y[in_coords[:, 0], :, in_coords[:, 1], in_coords[:, 2], in_coords[:, 3]]


def loop_ssc(coords, X, W, size, f):
    """SSC by seven nested loops over (site, offset, ci, co) -- tiny inputs only."""
    coords = [tuple(int(v) for v in r) for r in np.asarray(coords)]
    row = {c: i for i, c in enumerate(coords)}
    X = np.asarray(X, np.float64)
    W = np.asarray(W, np.float64)
    cin, cout = W.shape[1], W.shape[2]
    c = (f - 1) // 2
    Y = np.zeros((len(coords), cout))
    for k, (b, y0, y1, y2) in enumerate(coords):
        for i0 in range(f):
            for i1 in range(f):
                for i2 in range(f):
                    j = row.get((b, y0 + i0 - c, y1 + i1 - c, y2 + i2 - c))
                    if j is None:
                        continue
                    o = (i0 * f + i1) * f + i2
                    for ci in range(cin):
                        for co in range(cout):
                            Y[k, co] += X[j, ci] * W[o, ci, co]
    return Y


def active_in_field(coords, size, f, centred=True):
    """a = number of active inputs in each active site's f^3 field (Table 2)."""
    coords = np.asarray(coords, np.int64)
    B = int(coords[:, 0].max()) + 1
    occ = to_dense(coords, np.ones((coords.shape[0], 1)), size, B)
    cnt = F.conv3d(occ, torch.ones(1, 1, f, f, f, dtype=torch.float64),
                   padding=(f - 1) // 2 if centred else 0).numpy()[:, 0]
    return cnt[coords[:, 0], coords[:, 1], coords[:, 2], coords[:, 3]].astype(np.int64)


def dense_unet(coords, size, X, params, channels):
    """The U-Net of Sec. 5 on dense grids: every layer is a dense conv3d /
    conv_transpose3d in float64 followed by a mask that zeroes the inactive
    sites of the layer's output level (level l + 1 is active where a 2^3
    block of level l holds an active site); pre-activations are masked too,
    since an inactive site stays at the ground state 0.  Returns the features
    at the level-0 input sites, in input row order."""
    coords = np.asarray(coords, np.int64)
    B = int(coords[:, 0].max()) + 1
    depth = len(channels)
    masks = [to_dense(coords, np.ones((coords.shape[0], 1)), size, B)]
    for _ in range(depth - 1):
        masks.append((F.conv3d(masks[-1], torch.ones(1, 1, 2, 2, 2, dtype=torch.float64), stride=2) > 0).double())

    def pre(name, x, mask, k, cin, cout):
        scale, shift, W = params(name, k, cin, cout)
        sc = torch.from_numpy(np.asarray(scale, np.float64)).view(1, -1, 1, 1, 1)
        sh = torch.from_numpy(np.asarray(shift, np.float64)).view(1, -1, 1, 1, 1)
        return torch.relu(x * sc + sh) * mask, np.asarray(W, np.float64)

    def ssc(name, x, l, cin, cout):
        a, W = pre(name, x, masks[l], 27, cin, cout)
        return F.conv3d(a, torch_weight(W, 3), padding=1) * masks[l]

    def down(name, x, l):
        a, W = pre(name, x, masks[l], 8, channels[l], channels[l + 1])
        return F.conv3d(a, torch_weight(W, 2), stride=2) * masks[l + 1]

    def up(name, x, l):
        a, W = pre(name, x, masks[l + 1], 8, channels[l + 1], channels[l])
        w = torch.from_numpy(np.ascontiguousarray(W.reshape(2, 2, 2, channels[l + 1], channels[l]).transpose(3, 4, 0, 1, 2)))
        return F.conv_transpose3d(a, w, stride=2) * masks[l]

    x = to_dense(coords, X, size, B)
    skip = []
    for l in range(depth):
        x = ssc(f"enc{l}a", x, l, channels[l], channels[l])
        x = ssc(f"enc{l}b", x, l, channels[l], channels[l])
        skip.append(x)
        if l + 1 < depth:
            x = down(f"down{l}", x, l)
    for l in range(depth - 2, -1, -1):
        u = up(f"up{l}", x, l)
        x = torch.cat([skip[l], u], dim=1)
        x = ssc(f"dec{l}a", x, l, 2 * channels[l], channels[l])
        x = ssc(f"dec{l}b", x, l, channels[l], channels[l])
    y = x.numpy()
    return y[coords[:, 0], :, coords[:, 1], coords[:, 2], coords[:, 3]]


def dense_unet_train(coords, size, X, labels, params, channels, n_classes, eps=1e-5):
    """Loss and parameter gradients of the training step of the U-Net, on
    dense grids with torch autograd in float64.  Batch normalisation uses
    statistics over the active sites only (the masks); every activation is
    zeroed outside the active set of its level (the ground state 0); the head
    is batch normalisation + ReLU, a per-site linear layer with bias and the
    mean negative log-likelihood over the level-0 sites.  Returns
    (loss, {name: (dgamma, dbeta, dW[, db])}, {name: (mean, var)})."""
    coords = np.asarray(coords, np.int64)
    B = int(coords[:, 0].max()) + 1
    depth = len(channels)
    masks = [to_dense(coords, np.ones((coords.shape[0], 1)), size, B)]
    for _ in range(depth - 1):
        masks.append((F.conv3d(masks[-1], torch.ones(1, 1, 2, 2, 2, dtype=torch.float64), stride=2) > 0).double())
    leaves, stats = {}, {}

    def leaf(name, k, cin, cout):
        p = params(name, k, cin, cout)
        t = [torch.from_numpy(np.asarray(v, np.float64).copy()).requires_grad_(True) for v in p]
        leaves[name] = t
        return t

    def bn_relu(name, x, mask, gamma, beta):
        n = mask.sum()
        mean = (x * mask).sum(dim=(0, 2, 3, 4)) / n
        d = (x - mean.view(1, -1, 1, 1, 1)) * mask
        var = (d * d).sum(dim=(0, 2, 3, 4)) / n
        stats[name] = (mean.detach().numpy(), var.detach().numpy())
        xhat = d / torch.sqrt(var + eps).view(1, -1, 1, 1, 1)
        return torch.relu(gamma.view(1, -1, 1, 1, 1) * xhat + beta.view(1, -1, 1, 1, 1)) * mask

    def tw(W, f):
        K, cin, cout = W.shape
        return W.reshape(f, f, f, cin, cout).permute(4, 3, 0, 1, 2)

    def ssc(name, x, l, cin, cout):
        g, b, W = leaf(name, 27, cin, cout)
        return F.conv3d(bn_relu(name, x, masks[l], g, b), tw(W, 3), padding=1) * masks[l]

    def down(name, x, l):
        g, b, W = leaf(name, 8, channels[l], channels[l + 1])
        return F.conv3d(bn_relu(name, x, masks[l], g, b), tw(W, 2), stride=2) * masks[l + 1]

    def up(name, x, l):
        g, b, W = leaf(name, 8, channels[l + 1], channels[l])
        w = W.reshape(2, 2, 2, channels[l + 1], channels[l]).permute(3, 4, 0, 1, 2)
        return F.conv_transpose3d(bn_relu(name, x, masks[l + 1], g, b), w, stride=2) * masks[l]

    x = to_dense(coords, X, size, B)
    skip = []
    for l in range(depth):
        x = ssc(f"enc{l}a", x, l, channels[l], channels[l])
        x = ssc(f"enc{l}b", x, l, channels[l], channels[l])
        skip.append(x)
        if l + 1 < depth:
            x = down(f"down{l}", x, l)
    for l in range(depth - 2, -1, -1):
        u = up(f"up{l}", x, l)
        x = torch.cat([skip[l], u], dim=1)
        x = ssc(f"dec{l}a", x, l, 2 * channels[l], channels[l])
        x = ssc(f"dec{l}b", x, l, channels[l], channels[l])
    hg, hb, hW, hbias = leaf("head", 1, channels[0], n_classes)
    z = bn_relu("head", x, masks[0], hg, hb)
    zs = z[coords[:, 0], :, coords[:, 1], coords[:, 2], coords[:, 3]]      # active sites, input row order
    logits = zs @ hW[0] + hbias
    loss = F.cross_entropy(logits, torch.from_numpy(np.asarray(labels, np.int64)))
    loss.backward()
    grads = {k: tuple(t.grad.numpy().copy() for t in v) for k, v in leaves.items()}
    return float(loss.detach()), grads, stats


def dense_residual_block(coords, size, X, p1, p2, train=False, G=None, eps=1e-5):
    """A pre-activated residual block (two SSC(3) units, identity shortcut)
    on a dense grid in float64.  train: batch statistics over the active
    sites (masked), else inference affine maps.  With G (the gradient at the
    output, active rows), also returns the gradients by autograd.  Returns
    (Y at the active sites, grads or None)."""
    coords = np.asarray(coords, np.int64)
    B = int(coords[:, 0].max()) + 1
    mask = to_dense(coords, np.ones((coords.shape[0], 1)), size, B)
    x = to_dense(coords, X, size, B).requires_grad_(G is not None)
    ps = [[torch.from_numpy(np.asarray(v, np.float64).copy()).requires_grad_(G is not None) for v in p] for p in (p1, p2)]

    def pre(h, g, b):
        if not train:
            return torch.relu(h * g.view(1, -1, 1, 1, 1) + b.view(1, -1, 1, 1, 1)) * mask
        n = mask.sum()
        mean = (h * mask).sum(dim=(0, 2, 3, 4)) / n
        d = (h - mean.view(1, -1, 1, 1, 1)) * mask
        var = (d * d).sum(dim=(0, 2, 3, 4)) / n
        xh = d / torch.sqrt(var + eps).view(1, -1, 1, 1, 1)
        return torch.relu(g.view(1, -1, 1, 1, 1) * xh + b.view(1, -1, 1, 1, 1)) * mask

    def conv(a, W):
        K, cin, cout = W.shape
        return F.conv3d(a, W.reshape(3, 3, 3, cin, cout).permute(4, 3, 0, 1, 2), padding=1) * mask

    h = conv(pre(x, ps[0][0], ps[0][1]), ps[0][2])
    y = x + conv(pre(h, ps[1][0], ps[1][1]), ps[1][2])
    ys = y[coords[:, 0], :, coords[:, 1], coords[:, 2], coords[:, 3]]
    if G is None:
        return ys.detach().numpy(), None
    (ys * torch.from_numpy(np.asarray(G, np.float64))).sum().backward()
    gx = x.grad.numpy()[coords[:, 0], :, coords[:, 1], coords[:, 2], coords[:, 3]]
    return ys.detach().numpy(), (gx, tuple(t.grad.numpy() for t in ps[0]), tuple(t.grad.numpy() for t in ps[1]))


def dense_nd(coords, X, W, size, f, s, submanifold):
    """SSC / SC in d = 1, 2 or 4 dimensions on a dense grid (float64):
    conv1d / conv2d for d <= 2; for d = 4 the sum over the last filter axis
    of conv3d's of shifted 3-D slices.  Returns (active output coords in
    sorted order, features there)."""
    coords = np.asarray(coords, np.int64)
    d = len(size)
    B = int(coords[:, 0].max()) + 1
    X = np.asarray(X, np.float64)
    W = np.asarray(W, np.float64)
    K, cin, cout = W.shape
    dense = np.zeros((B, cin) + tuple(size))
    dense[(coords[:, 0], slice(None)) + tuple(coords[:, 1 + i] for i in range(d))] = X
    occ = np.zeros((B, 1) + tuple(size))
    occ[(coords[:, 0], 0) + tuple(coords[:, 1 + i] for i in range(d))] = 1.0
    w = W.reshape((f,) * d + (cin, cout))
    w = np.moveaxis(np.moveaxis(w, -1, 0), -1, 1)          # [cout][cin][i0]..[i_{d-1}]
    pad = (f - 1) // 2 if submanifold else 0
    stride = 1 if submanifold else s

    def conv(x, wt):
        xt, wtt = torch.from_numpy(np.ascontiguousarray(x)), torch.from_numpy(np.ascontiguousarray(wt))
        if d == 1:
            return F.conv1d(xt, wtt, padding=pad, stride=stride).numpy()
        if d == 2:
            return F.conv2d(xt, wtt, padding=pad, stride=stride).numpy()
        # d = 4: y[..., t] = sum_i3 conv3d(x[..., stride t + i3 - pad], w[..., i3])
        L3 = x.shape[-1]
        M3 = (L3 + 2 * pad - f) // stride + 1
        out = None
        for t in range(M3):
            acc = 0.0
            for i3 in range(f):
                src = stride * t + i3 - pad
                if 0 <= src < L3:
                    acc = acc + F.conv3d(torch.from_numpy(np.ascontiguousarray(x[..., src])),
                                         torch.from_numpy(np.ascontiguousarray(wt[..., i3])),
                                         padding=pad, stride=stride).numpy()
            if out is None:
                out = np.zeros(np.shape(acc) + (M3,))
            out[..., t] = acc
        return out

    y = conv(dense, w)
    if submanifold:
        act = coords[np.lexsort(tuple(coords[:, i] for i in range(d, -1, -1)))]
    else:
        cnt = conv(occ, np.ones((1, 1) + (f,) * d))[:, 0]
        act = np.argwhere(cnt > 0)
    vals = y[(act[:, 0], slice(None)) + tuple(act[:, 1 + i] for i in range(d))]
    return act.astype(np.int64), vals
