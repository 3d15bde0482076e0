"""Plant plausible mistakes in the CPU oracle and check that a pin catches each.

Mutations are applied with monkeypatch to the oracle module only (CPU), so
the oracle's pins are shown to be sensitive to: a sign error in the offset,
a dropped offset (term), a transposed weight operand, a wrong SSC centre, an
SC stride/offset mix-up and a backward that forgets an offset.
"""
import numpy as np
import pytest

from oracle import sscn_oracle as O
from tests import dense_ref as R


def _set(seed=1, size=(8, 8, 8)):
    rng = np.random.default_rng(seed)
    occ = rng.random((2,) + size) < 0.2
    b, x0, x1, x2 = np.nonzero(occ)
    return np.stack([b, x0, x1, x2], axis=1).astype(np.int32)


def _ssc_pin_error():
    size = (8, 8, 8)
    rng = np.random.default_rng(5)
    c = _set()
    X, W = rng.standard_normal((c.shape[0], 4)), rng.standard_normal((27, 4, 4))
    Y = O.forward(X, W, O.ssc_rulebook(c, size, 3))
    return np.abs(Y - R.dense_ssc(c, X, W, size, 3)).max()


def _sc_pin_error():
    size = (9, 9, 9)
    rng = np.random.default_rng(6)
    c = _set(size=size)
    X, W = rng.standard_normal((c.shape[0], 3)), rng.standard_normal((27, 3, 2))
    rb = O.sc_rulebook(c, size, 3, 2)
    act, vals, _ = R.dense_sc(c, X, W, size, 3, 2)
    if rb.n_out != act.shape[0]:
        return np.inf
    key = {tuple(r): i for i, r in enumerate(act.tolist())}
    try:
        idx = [key[tuple(r)] for r in rb.out_coords.tolist()]
    except KeyError:
        return np.inf
    return np.abs(O.forward(X, W, rb) - vals[idx]).max()


def _bwd_pin_error():
    size = (8, 8, 8)
    rng = np.random.default_rng(7)
    c = _set()
    X, W = rng.standard_normal((c.shape[0], 3)), rng.standard_normal((27, 3, 3))
    rb = O.ssc_rulebook(c, size, 3)
    G = rng.standard_normal((c.shape[0], 3))
    dX, dW = O.backward(X, W, G, rb)
    lhs = np.sum(O.forward(X, W, rb) * G)
    return max(abs(lhs - np.sum(X * dX)), abs(lhs - np.sum(W * dW)))


def _triples_pin_holds():
    from tests.test_oracle_pins import brute_force_triples
    rng = np.random.default_rng(8)
    size = (7, 7, 7)
    occ = rng.random((2,) + size) < 0.15
    c = np.argwhere(occ).astype(np.int32)
    c = c[rng.permutation(c.shape[0])]
    ok = True
    for rb, sub, f, s in ((O.ssc_rulebook(c, size, 3), True, 3, 1), (O.sc_rulebook(c, size, 3, 2), False, 3, 2)):
        want = brute_force_triples(c, rb.out_coords, f, s, sub)
        ok &= O.canonical_triples(rb).tolist() == [list(t) for t in want]
    return ok


def test_unmutated_pins_hold():
    assert _ssc_pin_error() < 1e-10
    assert _sc_pin_error() < 1e-10
    assert _bwd_pin_error() < 1e-10
    assert _triples_pin_holds()


@pytest.mark.parametrize("keys", [lambda t: (t[:, 1], t[:, 0], t[:, 2]),   # sorted by (o, in, out)
                                  lambda t: (t[:, 0], t[:, 2], t[:, 1]),   # sorted by (out, o, in)
                                  lambda t: (t[:, 2], t[:, 1], t[:, 0])])  # sorted by (in, out, o)
def test_triples_sort_key_caught(monkeypatch, keys):
    def bad(rb):
        t = np.concatenate([np.stack([rb.ins[o], rb.outs[o], np.full(rb.ins[o].size, o)], axis=1)
                            for o in range(rb.K)])
        return t[np.lexsort(keys(t))].astype(np.int64)
    monkeypatch.setattr(O, "canonical_triples", bad)
    assert not _triples_pin_holds()


def test_triples_swapped_columns_caught(monkeypatch):
    orig = O.canonical_triples
    monkeypatch.setattr(O, "canonical_triples", lambda rb: orig(rb)[:, [1, 0, 2]])
    assert not _triples_pin_holds()


def test_offset_sign_error_caught(monkeypatch):
    orig = O.filter_offsets
    monkeypatch.setattr(O, "filter_offsets", lambda f, d=3: (f - 1) - orig(f, d))
    assert _ssc_pin_error() > 1e-3


def test_dropped_offset_caught(monkeypatch):
    orig = O.ssc_rulebook

    def drop_last(*a):
        rb = orig(*a)
        rb.ins[-1] = rb.ins[-1][:0]
        rb.outs[-1] = rb.outs[-1][:0]
        return rb
    monkeypatch.setattr(O, "ssc_rulebook", drop_last)
    assert _ssc_pin_error() > 1e-3


def test_transposed_weight_caught(monkeypatch):
    orig = O.forward
    monkeypatch.setattr(O, "forward", lambda X, W, rb: orig(X, np.asarray(W).transpose(0, 2, 1), rb))
    assert _ssc_pin_error() > 1e-3


def test_wrong_ssc_centre_caught(monkeypatch):
    orig = O.filter_offsets
    # shifting the offsets by one voxel along x2 moves the SSC field off-centre
    monkeypatch.setattr(O, "filter_offsets", lambda f, d=3: orig(f, d) + np.eye(d, dtype=np.int64)[-1])
    assert _ssc_pin_error() > 1e-3


def test_sc_stride_mixup_caught(monkeypatch):
    orig = O.sc_output_size
    monkeypatch.setattr(O, "sc_output_size", lambda size, f, s: orig(size, f, 1) if s == 2 else orig(size, f, s))
    assert _sc_pin_error() > 1e-3


def test_backward_dropped_offset_caught(monkeypatch):
    orig = O.backward

    def bad(X, W, dY, rb):
        dX, dW = orig(X, W, dY, rb)
        dW[0] = 0.0
        return dX, dW
    monkeypatch.setattr(O, "backward", bad)
    assert _bwd_pin_error() > 1e-6


# --------------------------------------------------------------------------
# pooling and upsampling
# --------------------------------------------------------------------------
def _pool_pins_hold():
    from tests import test_oracle_pool as P
    try:
        for size, f, s in P.CASES:
            P.test_max_pool_is_relu_of_dense_max_pool(size, f, s)
            P.test_avg_pool_is_dense_avg_pool(size, f, s)
        P.test_max_pool_ties_go_to_the_smallest_offset()
        for size, s in [((8, 8, 8), 2), ((9, 9, 9), 3)]:
            P.test_upsample_is_dense_nearest(size, s)
    except AssertionError:
        return False
    return True


def test_pool_pins_hold_unmutated():
    assert _pool_pins_hold()


def test_max_pool_without_zero_floor_caught(monkeypatch):
    def bad(X, rb):
        X = np.asarray(X, np.float64)
        Y = np.full((rb.n_out, X.shape[1]), -np.inf)
        A = np.full((rb.n_out, X.shape[1]), O.NO_ARGMAX)
        for o in range(rb.K):
            j, k = rb.ins[o], rb.outs[o]
            win = X[j] > Y[k]
            Y[k] = np.where(win, X[j], Y[k])
            A[k] = np.where(win, o, A[k])
        return Y, A
    monkeypatch.setattr(O, "max_pool", bad)
    assert not _pool_pins_hold()


def test_max_pool_last_tie_caught(monkeypatch):
    orig = O.max_pool

    def bad(X, rb):
        # ties to the largest offset: run the offsets in reverse
        rb2 = O.Rulebook(rb.f, rb.stride, rb.submanifold, rb.n_in, rb.n_out, rb.in_size, rb.out_size,
                         rb.ins[::-1], rb.outs[::-1], rb.out_coords)
        Y, A = orig(X, rb2)
        return Y, np.where(A >= 0, rb.K - 1 - A, A)
    monkeypatch.setattr(O, "max_pool", bad)
    assert not _pool_pins_hold()


def test_avg_pool_by_count_caught(monkeypatch):
    def bad(X, rb):
        X = np.asarray(X, np.float64)
        Y = np.zeros((rb.n_out, X.shape[1]))
        cnt = np.zeros(rb.n_out)
        for o in range(rb.K):
            np.add.at(Y, rb.outs[o], X[rb.ins[o]])
            np.add.at(cnt, rb.outs[o], 1)
        return Y / cnt[:, None]
    monkeypatch.setattr(O, "avg_pool", bad)
    assert not _pool_pins_hold()


def test_upsample_wrong_parent_caught(monkeypatch):
    def bad(Y, rb):
        Y = np.asarray(Y, np.float64)
        out = np.zeros((rb.n_in, Y.shape[1]))
        for o in range(rb.K):
            out[rb.ins[o]] = Y[np.roll(rb.outs[o], 1)]      # each input gets another input's parent
        return out
    monkeypatch.setattr(O, "upsample_nearest", bad)
    assert not _pool_pins_hold()


# --------------------------------------------------------------------------
# training step
# --------------------------------------------------------------------------
def _train_pins_hold():
    from tests import test_oracle_train as T
    try:
        T.test_batch_norm_relu_is_torch_training_batch_norm()
        T.test_softmax_nll_is_cross_entropy()
        T.test_sgd_nesterov_is_torch_sgd()
        T.test_unet_train_step_matches_dense_autograd((3, 5))
    except AssertionError:
        return False
    return True


def test_train_pins_hold_unmutated():
    assert _train_pins_hold()


def test_bn_unbiased_variance_caught(monkeypatch):
    def bad(X, gamma, beta, eps=O.BN_EPS):
        X = np.asarray(X, np.float64)
        n = X.shape[0]
        mean = X.mean(axis=0)
        var = ((X - mean) ** 2).sum(axis=0) / (n - 1)
        return np.maximum(0.0, gamma * (X - mean) / np.sqrt(var + eps) + beta), mean, var
    monkeypatch.setattr(O, "batch_norm_relu_train", bad)
    assert not _train_pins_hold()


def test_bn_backward_without_relu_mask_caught(monkeypatch):
    orig = O.batch_norm_relu_backward

    def bad(dA, X, gamma, beta, mean, var, eps=O.BN_EPS):
        big = np.full_like(np.asarray(beta, np.float64), 1e6)   # every unit "active"
        return orig(dA, X, gamma, big, mean, var, eps)
    monkeypatch.setattr(O, "batch_norm_relu_backward", bad)
    assert not _train_pins_hold()


def test_bn_backward_missing_mean_term_caught(monkeypatch):
    orig = O.batch_norm_relu_backward

    def bad(dA, X, gamma, beta, mean, var, eps=O.BN_EPS):
        dX, dg, db = orig(dA, X, gamma, beta, mean, var, eps)
        n = np.asarray(X).shape[0]
        return dX + np.asarray(gamma) / np.sqrt(var + eps) / n * db, dg, db
    monkeypatch.setattr(O, "batch_norm_relu_backward", bad)
    assert not _train_pins_hold()


def test_plain_momentum_caught(monkeypatch):
    def bad(p, g, buf, lr, momentum=0.9, weight_decay=1e-4):
        g = np.asarray(g) + weight_decay * np.asarray(p)
        buf = momentum * np.asarray(buf) + g
        return np.asarray(p) - lr * buf, buf
    monkeypatch.setattr(O, "sgd_nesterov", bad)
    assert not _train_pins_hold()


def test_missing_weight_decay_caught(monkeypatch):
    orig = O.sgd_nesterov
    monkeypatch.setattr(O, "sgd_nesterov", lambda p, g, buf, lr, momentum=0.9, weight_decay=1e-4:
                        orig(p, g, buf, lr, momentum, 0.0))
    assert not _train_pins_hold()


def test_dropped_skip_gradient_caught(monkeypatch):
    orig = O.backward
    calls = {"n": 0}

    def bad(X, W, dY, rb):
        # the SC (down) layers' input gradients are lost, as if the skip
        # were the only consumer of each encoder output
        dX, dW = orig(X, W, dY, rb)
        if not rb.submanifold and rb.n_out < rb.n_in:
            dX = np.zeros_like(dX)
        return dX, dW
    monkeypatch.setattr(O, "backward", bad)
    assert not _train_pins_hold()


# --------------------------------------------------------------------------
# bias and residual blocks
# --------------------------------------------------------------------------
def _block_pins_hold():
    from tests import test_oracle_blocks as T
    try:
        for kind, f, s in (("ssc", 3, 1), ("sc", 2, 2)):
            T.test_forward_bias_is_dense_conv3d_with_bias(kind, f, s)
        T.test_residual_block_inference_is_dense()
        T.test_residual_block_training_matches_autograd()
    except AssertionError:
        return False
    return True


def test_block_pins_hold_unmutated():
    assert _block_pins_hold()


def test_bias_dropped_caught(monkeypatch):
    monkeypatch.setattr(O, "forward_bias", lambda X, W, b, rb: O.forward(X, W, rb))
    assert not _block_pins_hold()


def test_residual_without_shortcut_gradient_caught(monkeypatch):
    orig = O.residual_block_train_backward

    def bad(dY, cache):
        dX, g1, g2 = orig(dY, cache)
        return dX - np.asarray(dY), g1, g2
    monkeypatch.setattr(O, "residual_block_train_backward", bad)
    assert not _block_pins_hold()


# --------------------------------------------------------------------------
# other dimensions
# --------------------------------------------------------------------------
def _nd_pins_hold():
    from tests import test_oracle_nd as T
    try:
        for case in T.CASES:
            T.test_nd_rulebook_and_forward(*case)
        T.test_4d_with_one_position_on_the_last_axis_is_3d(3, 1, True)
        T.test_4d_with_one_position_on_the_last_axis_is_3d(2, 2, False)
    except (AssertionError, O.OracleError):   # a planted mistake may also make the oracle refuse the input
        return False
    return True


def test_nd_pins_hold_unmutated():
    assert _nd_pins_hold()


def test_nd_offset_order_reversed_caught(monkeypatch):
    orig = O.filter_offsets
    monkeypatch.setattr(O, "filter_offsets", lambda f, d=3: orig(f, d)[:, ::-1].copy())
    assert not _nd_pins_hold()


def test_nd_key_ignoring_an_axis_caught(monkeypatch):
    orig = O.location_key
    monkeypatch.setattr(O, "location_key", lambda coords, size: orig(np.asarray(coords)[:, :-1], size[:-1])
                        if len(size) == 4 else orig(coords, size))
    assert not _nd_pins_hold()
