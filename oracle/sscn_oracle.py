"""CPU oracle for sparse (SC) and submanifold sparse (SSC) convolutions.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path imports this module:
only the test-suite, the smoke check and the CPU-baseline leg of the
benchmark may call it.  It shares no code with the GPU library.

It is a plain, slow, fp64 transcription of the paper's definitions
(Graham, Engelcke & van der Maaten, "3D Semantic Segmentation with
Submanifold Sparse Convolutional Networks", arXiv:1711.10275):

* feature matrix + (location -> row) dictionary                 Sec. 4.2
* filter offsets F = {0..f-1}^d and a rule book R = (R_i)       Sec. 4.2
* SC(m, n, f, s): output active iff the f^d field holds an active
  input; output size (l - f + s) / s; inactive inputs read as 0  Sec. 4.1
* SSC(m, n, f): f odd, pad (f-1)/2, output active iff the centre
  input is active, i.e. the output set is the input set         Sec. 4.1
* DC: the SC connections inverted; output set = SC input set    Sec. 4.1
* output = 0, then out[k] += in[j] W^i for every (j, k) in R_i   Sec. 4.2
* MP / AP pooling over SC connections, nearest-neighbour
  upsampling back through them                   Sec. 4.1, Sec. 5
* backward: the adjoint of that linear map (the paper trains the
  networks, Sec. 6.2, but does not spell the gradients out)

Readings where the paper leaves a choice open (each is listed in the design
notes of the repository):

* offsets are enumerated o = i0*f^2 + i1*f + i2 (first coordinate most
  significant); the SSC centre is o = (f^3 - 1) / 2;
* the operation is a cross-correlation: an SSC output at y reads the input
  at y + i - (f-1)/2, an SC output at y reads the input at s*y + i;
* SC outputs are numbered in the order of their first visit when the input
  rows are iterated in row order and, for each input, the filter offsets in
  the order above (Sec. 4.2 step 1 with the iteration order fixed);
* (L - f) must be divisible by s and L >= f (else a shape error);
* the batch index is part of the location, so samples never interact;
* two rows at one location is an error (one row per active site);
* ground state 0; a bias term, where a layer has one, is added to every
  active output row (inactive sites are not stored);
* MP ties go to the smallest offset; AP divides by f^d whatever the number
  of active inputs; nearest-neighbour upsampling inverts an SC(s, s);
* batch normalisation in training form normalises with the biased variance
  over the active rows (eps 1e-5) and keeps running statistics with
  momentum 0.1 and the unbiased variance.

Only numpy is used; the dictionary is a sorted key array searched with
numpy.searchsorted, and each per-offset product is one numpy matmul.
"""
from __future__ import annotations

import dataclasses
import itertools

import numpy as np

D = 3  # spatial dimensions unless a layer's grid says otherwise


class OracleError(Exception):
    code = "invalid_arg"


class InvalidArg(OracleError):
    code = "invalid_arg"


class ShapeError(OracleError):
    code = "shape"


class OutOfRange(OracleError):
    code = "out_of_range"


class Duplicate(OracleError):
    code = "duplicate"


MAX_BATCH = 1 << 15
MAX_EXTENT = 1 << 16


def filter_offsets(f, d=D):
    """F = {0..f-1}^d as an (f^d, d) array in lexicographic order (first
    coordinate most significant): for d = 3, row o = (o // f^2, (o // f) % f, o % f)."""
    return np.array(list(itertools.product(range(f), repeat=d)), dtype=np.int64).reshape(-1, d)


def location_key(coords, size):
    """One integer per location (b, x_0, .., x_{d-1}) inside a grid of extent `size`."""
    c = np.asarray(coords, np.int64)
    key = c[:, 0].copy()
    for dd, L in enumerate(size):
        key = key * int(L) + c[:, 1 + dd]
    return key


class CoordTable:
    """The (location -> row) dictionary of Sec. 4.2 for one layer's active sites."""

    def __init__(self, coords, size):
        coords = np.asarray(coords)
        if coords.ndim != 2 or coords.shape[1] != len(size) + 1:
            raise InvalidArg("coords must be n x (d + 1) for a d-dimensional grid")
        c = coords.astype(np.int64)
        size = tuple(int(v) for v in size)
        if any(v < 1 or v > MAX_EXTENT for v in size):
            raise InvalidArg("spatial size out of range")
        if c.shape[0]:
            if (c[:, 0].min() < 0 or c[:, 0].max() >= MAX_BATCH
                    or np.any(c[:, 1:] < 0) or np.any(c[:, 1:] >= np.array(size))):
                raise OutOfRange("coordinate outside the grid")
        self.size = size
        self.coords = c
        keys = location_key(c, size)
        order = np.argsort(keys, kind="stable")
        self.sorted_keys = keys[order]
        self.sorted_rows = order
        if np.any(self.sorted_keys[1:] == self.sorted_keys[:-1]):
            raise Duplicate("two rows share one location")

    def lookup(self, query):
        """Row of each queried location, -1 where the location is not active."""
        q = np.asarray(query, np.int64)
        out = np.full(q.shape[0], -1, np.int64)
        inside = np.all((q[:, 1:] >= 0) & (q[:, 1:] < np.array(self.size)), axis=1)
        if not np.any(inside) or self.sorted_keys.size == 0:
            return out
        k = location_key(q[inside], self.size)
        pos = np.searchsorted(self.sorted_keys, k)
        pos_c = np.minimum(pos, self.sorted_keys.size - 1)
        hit = self.sorted_keys[pos_c] == k
        rows = np.where(hit, self.sorted_rows[pos_c], -1)
        out[inside] = rows
        return out


@dataclasses.dataclass
class Rulebook:
    """R = (R_o : o in F), each R_o a pair of equal-length row arrays (in, out)."""
    f: int
    stride: int
    submanifold: bool
    n_in: int
    n_out: int
    in_size: tuple
    out_size: tuple
    ins: list            # K arrays of input rows
    outs: list           # K arrays of output rows
    out_coords: np.ndarray  # n_out x (d + 1) int64

    @property
    def d(self):
        return len(self.in_size)

    @property
    def K(self):
        return self.f ** self.d

    def pairs_per_offset(self):
        return np.array([a.size for a in self.ins], np.int64)

    def n_pairs(self):
        return int(sum(a.size for a in self.ins))


def ssc_rulebook(coords, size, f):
    """SSC(., ., f) rule book (Sec. 4.1 definition, Sec. 4.2 construction).

    The input dictionary serves as the output dictionary; for every active
    site k and offset i in F the neighbour at x_k + i - (f-1)/2 is looked up,
    and a hit j adds the row (j, k) to R_i.
    """
    if f < 1 or f % 2 == 0:
        raise InvalidArg("SSC needs an odd filter size")
    table = CoordTable(coords, size)
    c = table.coords
    centre = (f - 1) // 2
    ins, outs = [], []
    for i in filter_offsets(f, len(table.size)):
        q = c.copy()
        q[:, 1:] += i - centre
        j = table.lookup(q)
        k = np.nonzero(j >= 0)[0]
        ins.append(j[k])
        outs.append(k)
    n = c.shape[0]
    return Rulebook(f, 1, True, n, n, table.size, table.size, ins, outs, c.copy())


def sc_output_size(size, f, s):
    """Output extent (l - f + s) / s per dimension (Sec. 4.1)."""
    if f < 1 or s < 1:
        raise InvalidArg("filter size and stride must be positive")
    out = []
    for L in size:
        if L < f or (L - f) % s != 0:
            raise ShapeError("(L - f) must be a non-negative multiple of s")
        out.append((L - f + s) // s)
    return tuple(out)


def sc_rulebook(coords, size, f, s):
    """SC(., ., f, s) rule book built in one pass over the inputs (Sec. 4.2).

    Input rows are visited in row order, and for each input x the outputs y
    that see it are visited in offset order: x = s*y + i for i in F.  An
    output site gets the next free row at its first visit, and the pair
    (row(x), row(y)) is appended to R_i.
    """
    size = tuple(int(v) for v in size)
    out_size = sc_output_size(size, f, s)
    table = CoordTable(coords, size)
    c = table.coords
    d = len(size)
    n, F = c.shape[0], filter_offsets(f, d)
    K = F.shape[0]
    # visit (j, o): y = (x_j - i_o) / s when that is integral and inside the output grid
    t = c[:, None, 1:] - F[None, :, :]                        # n x K x 3
    valid = np.all((t % s == 0) & (t >= 0) & (t // s < np.array(out_size)), axis=2)
    y = t // s
    b = np.broadcast_to(c[:, None, 0:1], (n, K, 1))
    ycoords = np.concatenate([b, y], axis=2).reshape(n * K, d + 1)
    vflat = valid.reshape(n * K)
    visit = np.nonzero(vflat)[0]                              # visit order = (j, o) lexicographic
    keys = location_key(ycoords[visit], out_size)
    # first visit of each output location -> output row in order of first visit
    uniq, first = np.unique(keys, return_index=True)
    order = np.argsort(first, kind="stable")
    row_of_uniq = np.empty(uniq.size, np.int64)
    row_of_uniq[order] = np.arange(uniq.size)
    out_rows = row_of_uniq[np.searchsorted(uniq, keys)]
    out_coords = ycoords[visit[first[order]]]
    j_of_visit, o_of_visit = visit // K, visit % K
    ins, outs = [], []
    for o in range(K):
        m = o_of_visit == o
        ins.append(j_of_visit[m])
        outs.append(out_rows[m])
    return Rulebook(f, s, False, n, int(uniq.size), size, out_size, ins, outs, out_coords)


def transpose(rb):
    """DC connectivity (Sec. 4.1): the same pairs with input and output swapped."""
    return Rulebook(rb.f, rb.stride, rb.submanifold, rb.n_out, rb.n_in, rb.out_size, rb.in_size,
                    [a.copy() for a in rb.outs], [a.copy() for a in rb.ins], None)


def forward(X, W, rb):
    """out = 0; out[k] += X[j] @ W[o] for every (j, k) in R_o (Sec. 4.2 step 2), fp64."""
    X = np.asarray(X, np.float64)
    W = np.asarray(W, np.float64)
    if W.shape[0] != rb.K or X.shape[0] != rb.n_in or W.shape[1] != X.shape[1]:
        raise ShapeError("shape mismatch")
    Y = np.zeros((rb.n_out, W.shape[2]), np.float64)
    for o in range(rb.K):
        if rb.ins[o].size:
            np.add.at(Y, rb.outs[o], X[rb.ins[o]] @ W[o])
    return Y


def backward(X, W, dY, rb):
    """Adjoint of `forward`: dX[j] += dY[k] @ W[o]^T, dW[o] += X[j]^T dY[k], fp64."""
    X = np.asarray(X, np.float64)
    W = np.asarray(W, np.float64)
    dY = np.asarray(dY, np.float64)
    dX = np.zeros_like(X)
    dW = np.zeros_like(W)
    for o in range(rb.K):
        j, k = rb.ins[o], rb.outs[o]
        if j.size:
            np.add.at(dX, j, dY[k] @ W[o].T)
            dW[o] = X[j].T @ dY[k]
    return dX, dW


def forward_bias(X, W, b, rb):
    """A convolution with a bias term (Sec. 3 footnote): forward(X, W, rb)
    plus b on every active output row.  Inactive sites are not stored, so
    the ground state the bias would give them does not appear."""
    return forward(X, W, rb) + np.asarray(b, np.float64)


def canonical_triples(rb):
    """All pairs as (in, out, o) rows sorted by (o, out, in)."""
    if rb.n_pairs() == 0:
        return np.zeros((0, 3), np.int64)
    t = np.concatenate([np.stack([rb.ins[o], rb.outs[o], np.full(rb.ins[o].size, o)], axis=1)
                        for o in range(rb.K)])
    order = np.lexsort((t[:, 0], t[:, 1], t[:, 2]))
    return t[order].astype(np.int64)


def macs(rb, cin, cout):
    """Multiply-adds of one layer: sum over output sites of a*m*n (Table 2)."""
    return rb.n_pairs() * cin * cout


# --------------------------------------------------------------------------
# pooling and upsampling (Sec. 4.1 "Other operators"; Sec. 5 FCN upsampling)
# --------------------------------------------------------------------------
NO_ARGMAX = -1   # the zero vector is the maximum (no input receives gradient)


def _pool_rulebook(rb):
    if rb.submanifold:
        raise InvalidArg("pooling is defined over SC(f, s) connections")
    return rb


def max_pool(X, rb):
    """MP(f, s): a variant of SC(., ., f, s) whose output at each active site
    is, per channel, the maximum of the zero vector and the input vectors in
    its receptive field (Sec. 4.1).  rb is the SC(f, s) rule book.

    Returns (Y, A): Y n_out x C (fp64) and A n_out x C, the offset o of the
    input that attains each maximum (the smallest such o when several tie),
    or NO_ARGMAX where no input exceeds zero."""
    _pool_rulebook(rb)
    X = np.asarray(X, np.float64)
    C = X.shape[1]
    Y = np.zeros((rb.n_out, C), np.float64)
    A = np.full((rb.n_out, C), NO_ARGMAX, np.int64)
    for o in range(rb.K):                   # increasing o: a later equal value never wins
        j, k = rb.ins[o], rb.outs[o]        # within one R_o every output appears once
        v = X[j]
        win = v > Y[k]
        Y[k] = np.where(win, v, Y[k])
        A[k] = np.where(win, o, A[k])
    return Y, A


def max_pool_backward(dY, A, rb):
    """Gradient of max_pool: each output element's gradient goes to the
    input that attained its maximum (none where the zero vector did)."""
    _pool_rulebook(rb)
    dY = np.asarray(dY, np.float64)
    dX = np.zeros((rb.n_in, dY.shape[1]), np.float64)
    for o in range(rb.K):
        j, k = rb.ins[o], rb.outs[o]
        np.add.at(dX, j, np.where(A[k] == o, dY[k], 0.0))
    return dX


def avg_pool(X, rb):
    """AP(f, s): f^-d times the sum of the active input vectors in the
    receptive field (Sec. 4.1); inactive sites contribute zero."""
    _pool_rulebook(rb)
    X = np.asarray(X, np.float64)
    Y = np.zeros((rb.n_out, X.shape[1]), np.float64)
    for o in range(rb.K):
        np.add.at(Y, rb.outs[o], X[rb.ins[o]])
    return Y / float(rb.K)


def avg_pool_backward(dY, rb):
    _pool_rulebook(rb)
    dY = np.asarray(dY, np.float64)
    dX = np.zeros((rb.n_in, dY.shape[1]), np.float64)
    for o in range(rb.K):
        np.add.at(dX, rb.ins[o], dY[rb.outs[o]])
    return dX / float(rb.K)


def upsample_nearest(Y, rb):
    """Nearest-neighbour upsampling of the FCN (Sec. 5): features on the
    output sites of an SC(s, s) downsampling are copied back to every input
    site of it, i.e. input site x receives the features of the output site
    whose s^d block holds x.  Needs f = s (each input has exactly one such
    output)."""
    if rb.submanifold or rb.f != rb.stride:
        raise InvalidArg("nearest-neighbour upsampling inverts an SC(s, s) downsampling")
    Y = np.asarray(Y, np.float64)
    out = np.zeros((rb.n_in, Y.shape[1]), np.float64)
    for o in range(rb.K):
        out[rb.ins[o]] = Y[rb.outs[o]]
    return out


def upsample_nearest_backward(dOut, rb):
    """Gradient of upsample_nearest: each output site sums the gradients of
    the input sites it was copied to."""
    if rb.submanifold or rb.f != rb.stride:
        raise InvalidArg("nearest-neighbour upsampling inverts an SC(s, s) downsampling")
    dOut = np.asarray(dOut, np.float64)
    dY = np.zeros((rb.n_out, dOut.shape[1]), np.float64)
    for o in range(rb.K):
        np.add.at(dY, rb.outs[o], dOut[rb.ins[o]])
    return dY


# --------------------------------------------------------------------------
# network pieces (Sec. 5): pre-activation, row-sampled layers, the U-Net
# --------------------------------------------------------------------------
def affine_relu(X, scale, shift):
    """max(0, x * scale + shift) per channel on the active rows (inference-form
    batch normalisation followed by ReLU; inactive sites are not stored, so
    they keep the ground state 0, Sec. 4.1), fp64."""
    X = np.asarray(X, np.float64)
    return np.maximum(0.0, X * np.asarray(scale, np.float64) + np.asarray(shift, np.float64))


def forward_rows(X, W, rb, rows):
    """Rows `rows` of forward(X, W, rb): for each requested output site, the
    sum over the pairs (j, k) of every R_o that reach it (Sec. 4.2 step 2)."""
    X = np.asarray(X, np.float64)
    W = np.asarray(W, np.float64)
    rows = np.asarray(rows, np.int64)
    pos = np.full(rb.n_out, -1, np.int64)
    pos[rows] = np.arange(rows.size)
    Y = np.zeros((rows.size, W.shape[2]), np.float64)
    for o in range(rb.K):
        p = pos[rb.outs[o]]
        m = p >= 0
        if m.any():
            np.add.at(Y, p[m], X[rb.ins[o][m]] @ W[o])
    return Y


def round_bf16(a):
    """Nearest bfloat16 value (8 significant bits, ties to even) of each
    finite element, returned as float64."""
    a = np.asarray(a, np.float64)
    m, e = np.frexp(a)                      # a = m 2^e, 0.5 <= |m| < 1
    return np.ldexp(np.round(m * 256.0) / 256.0, e)


def unet_forward(coords, size, X, params, channels, round_to_bf16=True):
    """Submanifold U-Net of Sec. 5 on level-0 sites `coords`.

    Levels l = 0 .. len(channels) - 1 with C_l = channels[l].  Encoder: two
    pre-activated SSC(3) units C_l -> C_l per level (the result is the skip
    of level l), then a pre-activated SC(2, 2) unit C_l -> C_{l+1} to the
    next level.  Decoder, from the second-lowest level up: a pre-activated
    DC unit C_{l+1} -> C_l over the inverted SC connections, the skip and
    the upsampled features side by side (skip first), and two
    pre-activated SSC(3) units 2 C_l -> C_l and C_l -> C_l.

    params(name, k, cin, cout) -> (scale, shift, W) for the units named
    enc{l}a, enc{l}b, down{l}, up{l}, dec{l}a, dec{l}b.  With
    round_to_bf16 every stored activation (pre-activated input and
    convolution output) is rounded to bfloat16, as a bf16 network stores
    them; the arithmetic itself is fp64.
    """
    rnd = round_bf16 if round_to_bf16 else (lambda a: a)
    depth = len(channels)

    def unit(name, x, rb, cin, cout):
        scale, shift, W = params(name, rb.K, cin, cout)
        return rnd(forward(rnd(affine_relu(x, scale, shift)), W, rb))

    ssc_rb, sc_rb = [], []
    c, sz = np.asarray(coords), tuple(size)
    for l in range(depth):
        ssc_rb.append(ssc_rulebook(c, sz, 3))
        if l + 1 < depth:
            sc_rb.append(sc_rulebook(c, sz, 2, 2))
            c, sz = sc_rb[-1].out_coords, sc_rb[-1].out_size

    x = rnd(np.asarray(X, np.float64))
    skip = []
    for l in range(depth):
        x = unit(f"enc{l}a", x, ssc_rb[l], channels[l], channels[l])
        x = unit(f"enc{l}b", x, ssc_rb[l], channels[l], channels[l])
        skip.append(x)
        if l + 1 < depth:
            x = unit(f"down{l}", x, sc_rb[l], channels[l], channels[l + 1])
    for l in range(depth - 2, -1, -1):
        up = unit(f"up{l}", x, transpose(sc_rb[l]), channels[l + 1], channels[l])
        x = np.concatenate([skip[l], up], axis=1)
        x = unit(f"dec{l}a", x, ssc_rb[l], 2 * channels[l], channels[l])
        x = unit(f"dec{l}b", x, ssc_rb[l], channels[l], channels[l])
    return x


# --------------------------------------------------------------------------
# training (Sec. 4.1: batch normalisation over the active sites, ReLU on
# them; Sec. 5: pre-activated units, a per-site linear layer and softmax;
# Sec. 6.2: negative log-likelihood, SGD with Nesterov momentum and L2
# weight decay)
# --------------------------------------------------------------------------
BN_EPS = 1e-5
BN_MOMENTUM = 0.1


def batch_norm_relu_train(X, gamma, beta, eps=BN_EPS):
    """relu(gamma (x - mean) / sqrt(var + eps) + beta) per channel, with the
    mean and the (biased) variance taken over the active rows: regular batch
    normalisation applied to the set of active sites (Sec. 4.1).  Returns
    (A, mean, var)."""
    X = np.asarray(X, np.float64)
    n = X.shape[0]
    mean = X.sum(axis=0) / n
    var = ((X - mean) ** 2).sum(axis=0) / n
    xhat = (X - mean) / np.sqrt(var + eps)
    return np.maximum(0.0, np.asarray(gamma, np.float64) * xhat + np.asarray(beta, np.float64)), mean, var


def batch_norm_relu_backward(dA, X, gamma, beta, mean, var, eps=BN_EPS):
    """Gradients (dX, dgamma, dbeta) of batch_norm_relu_train at its input X,
    given dA, the gradient at its output."""
    X = np.asarray(X, np.float64)
    gamma = np.asarray(gamma, np.float64)
    n = X.shape[0]
    invstd = 1.0 / np.sqrt(var + eps)
    xhat = (X - mean) * invstd
    dz = np.where(gamma * xhat + np.asarray(beta, np.float64) > 0.0, np.asarray(dA, np.float64), 0.0)
    dbeta = dz.sum(axis=0)
    dgamma = (dz * xhat).sum(axis=0)
    dX = gamma * invstd / n * (n * dz - dbeta - xhat * dgamma)
    return dX, dgamma, dbeta


def running_stats(running_mean, running_var, mean, var, n, momentum=BN_MOMENTUM):
    """The inference statistics after one training step: exponential moving
    averages of the batch mean and the unbiased batch variance."""
    unbiased = var * n / max(n - 1, 1)
    return ((1.0 - momentum) * np.asarray(running_mean, np.float64) + momentum * mean,
            (1.0 - momentum) * np.asarray(running_var, np.float64) + momentum * unbiased)


def softmax_nll(logits, labels):
    """Mean over the active sites of -log softmax(logits)[label], and its
    gradient with respect to the logits."""
    z = np.asarray(logits, np.float64)
    labels = np.asarray(labels, np.int64)
    n = z.shape[0]
    m = z.max(axis=1, keepdims=True)
    e = np.exp(z - m)
    ssum = e.sum(axis=1, keepdims=True)
    logp = z - m - np.log(ssum)
    loss = -logp[np.arange(n), labels].sum() / n
    d = e / ssum
    d[np.arange(n), labels] -= 1.0
    return loss, d / n


def sgd_nesterov(p, g, buf, lr, momentum=0.9, weight_decay=1e-4):
    """One SGD step with Nesterov momentum and L2 weight decay (Sec. 6.2):
    g' = g + wd p; buf' = momentum buf + g'; p' = p - lr (g' + momentum buf').
    buf starts at zero.  Returns (p', buf')."""
    p = np.asarray(p, np.float64)
    g = np.asarray(g, np.float64) + weight_decay * p
    buf = momentum * np.asarray(buf, np.float64) + g
    return p - lr * (g + momentum * buf), buf


def unet_train_step(coords, size, X, labels, params, channels, n_classes):
    """Loss and parameter gradients of one training step of the U-Net of
    unet_forward, with every unit's batch normalisation in training form
    (batch statistics of its input over the active sites) and a head on the
    level-0 output: batch normalisation + ReLU, then a per-site linear layer
    (an SSC(C_0, n_classes, 1) convolution plus a bias) and softmax, scored
    by the mean negative log-likelihood of `labels` (one class per input
    site).  fp64 throughout.

    params(name, k, cin, cout) -> (gamma, beta, W) for every unit, and for
    name "head" (k = 1, cin = C_0, cout = n_classes) -> (gamma, beta, W, b).
    Returns (loss, grads, stats): grads[name] = (dgamma, dbeta, dW) and
    grads["head"] = (dgamma, dbeta, dW, db); stats[name] = (mean, var) of
    each batch normalisation."""
    depth = len(channels)
    ssc_rb, sc_rb = [], []
    c, sz = np.asarray(coords), tuple(size)
    for l in range(depth):
        ssc_rb.append(ssc_rulebook(c, sz, 3))
        if l + 1 < depth:
            sc_rb.append(sc_rulebook(c, sz, 2, 2))
            c, sz = sc_rb[-1].out_coords, sc_rb[-1].out_size

    tape = []                                   # (name, rb, x, a, W, gamma, beta, mean, var)
    stats = {}

    def unit(name, x, rb, cin, cout):
        gamma, beta, W = params(name, rb.K, cin, cout)
        a, mean, var = batch_norm_relu_train(x, gamma, beta)
        stats[name] = (mean, var)
        tape.append((name, rb, x, a, W, gamma, beta, mean, var))
        return forward(a, W, rb)

    x = np.asarray(X, np.float64)
    skip = []
    for l in range(depth):
        x = unit(f"enc{l}a", x, ssc_rb[l], channels[l], channels[l])
        x = unit(f"enc{l}b", x, ssc_rb[l], channels[l], channels[l])
        skip.append(x)
        if l + 1 < depth:
            x = unit(f"down{l}", x, sc_rb[l], channels[l], channels[l + 1])
    for l in range(depth - 2, -1, -1):
        up = unit(f"up{l}", x, transpose(sc_rb[l]), channels[l + 1], channels[l])
        x = np.concatenate([skip[l], up], axis=1)
        x = unit(f"dec{l}a", x, ssc_rb[l], 2 * channels[l], channels[l])
        x = unit(f"dec{l}b", x, ssc_rb[l], channels[l], channels[l])
    hg, hb, hW, hbias = params("head", 1, channels[0], n_classes)
    h1 = ssc_rulebook(coords, size, 1)
    z, hmean, hvar = batch_norm_relu_train(x, hg, hb)
    stats["head"] = (hmean, hvar)
    logits = forward(z, hW, h1) + np.asarray(hbias, np.float64)
    loss, dlogits = softmax_nll(logits, labels)

    grads = {}
    dz, dhW = backward(z, hW, dlogits, h1)
    dx, dhg, dhb = batch_norm_relu_backward(dz, x, hg, hb, hmean, hvar)
    grads["head"] = (dhg, dhb, dhW, dlogits.sum(axis=0))

    def unit_back(dy):
        name, rb, xin, a, W, gamma, beta, mean, var = tape.pop()
        da, dW = backward(a, W, dy, rb)
        dxin, dg, db = batch_norm_relu_backward(da, xin, gamma, beta, mean, var)
        grads[name] = (dg, db, dW)
        return name, dxin

    dskip = {}
    for l in range(depth - 1):
        _, dx = unit_back(dx)                   # dec{l}b
        _, dcat = unit_back(dx)                 # dec{l}a
        C = channels[l]
        dskip[l] = dcat[:, :C]
        _, dx = unit_back(dcat[:, C:])          # up{l}: gradient at level l + 1
    for l in range(depth - 1, -1, -1):
        if l + 1 < depth:
            _, dx = unit_back(dx)               # down{l}: into enc{l}b's output ...
            dx = dx + dskip.pop(l)              # ... which also feeds the concatenation
        _, dx = unit_back(dx)                   # enc{l}b
        _, dx = unit_back(dx)                   # enc{l}a
    assert not tape
    return loss, grads, stats


# --------------------------------------------------------------------------
# pre-activated residual blocks (Sec. 5): two SSC(3) units and an identity
# shortcut, same number of input and output features
# --------------------------------------------------------------------------
def residual_block(X, rb, p1, p2):
    """Inference form: X + SSC(relu(affine2(SSC(relu(affine1(X)), W1))), W2)
    with p = (scale, shift, W) per unit; rb is the level's SSC(3) rule book."""
    s1, t1, W1 = p1
    s2, t2, W2 = p2
    h = forward(affine_relu(X, s1, t1), W1, rb)
    return np.asarray(X, np.float64) + forward(affine_relu(h, s2, t2), W2, rb)


def residual_block_train(X, rb, p1, p2):
    """Training form (batch statistics in both normalisations), p = (gamma,
    beta, W).  Returns (Y, cache) for residual_block_train_backward."""
    X = np.asarray(X, np.float64)
    g1, b1, W1 = p1
    g2, b2, W2 = p2
    a1, m1, v1 = batch_norm_relu_train(X, g1, b1)
    h = forward(a1, W1, rb)
    a2, m2, v2 = batch_norm_relu_train(h, g2, b2)
    return X + forward(a2, W2, rb), (X, rb, p1, p2, a1, m1, v1, h, a2, m2, v2)


def residual_block_train_backward(dY, cache):
    """Gradients of residual_block_train: (dX, (dgamma1, dbeta1, dW1),
    (dgamma2, dbeta2, dW2)).  The shortcut passes dY to X unchanged."""
    X, rb, (g1, b1, W1), (g2, b2, W2), a1, m1, v1, h, a2, m2, v2 = cache
    dY = np.asarray(dY, np.float64)
    da2, dW2 = backward(a2, W2, dY, rb)
    dh, dg2, db2 = batch_norm_relu_backward(da2, h, g2, b2, m2, v2)
    da1, dW1 = backward(a1, W1, dh, rb)
    dX, dg1, db1 = batch_norm_relu_backward(da1, X, g1, b1, m1, v1)
    return dY + dX, (dg1, db1, dW1), (dg2, db2, dW2)
