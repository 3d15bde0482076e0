"""The training step on the GPU against the oracle: the batch-statistics
normalisation and its gradients, softmax / negative log-likelihood, the
Nesterov SGD update, bias and residual helpers, and one whole step of the
U-Net (every parameter gradient, the loss, the running statistics and the
updated parameters)."""
import numpy as np
import pytest
import torch

from oracle import sscn_oracle as O
from paper_1711_10275_amd import sscn, train, unet
from paper_1711_10275_amd import synthetic as S
from tests.gpu_common import dev, host
from tests.parity import assert_close

pytestmark = pytest.mark.gpu

TD = {"f32": torch.float32, "bf16": torch.bfloat16}


def _mat(rng, n, c, dtype, loc=0.0, scale=1.0):
    x = (rng.standard_normal((n, c)) * scale + loc).astype(np.float32)
    return S.bf16_round(x) if dtype == "bf16" else x


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("n,c", [(1, 3), (777, 5), (20000, 64), (100003, 70)])
def test_batchnorm_forward_backward(n, c, dtype):
    rng = np.random.default_rng(n + c)
    x = _mat(rng, n, c, dtype, loc=2.0, scale=3.0)
    g = rng.uniform(0.5, 1.5, c).astype(np.float32)
    b = rng.normal(0, 0.5, c).astype(np.float32)
    rm, rv = torch.zeros(c, device="cuda:0"), torch.ones(c, device="cuda:0")
    tx = dev(x, TD[dtype])
    st = sscn.batchnorm_forward(tx, dev(g), dev(b), running_mean=rm, running_var=rv)
    a = sscn.batchnorm_relu_apply(tx, st, dev(b))
    A, mean, var = O.batch_norm_relu_train(x, g, b)
    assert_close(host(st.mean), mean, "f32", "mean")
    assert_close(host(st.invstd), 1 / np.sqrt(var + O.BN_EPS), "f32", "invstd")
    assert_close(host(a), A, dtype, "bn-relu")
    em, ev = O.running_stats(np.zeros(c), np.ones(c), mean, var, n)
    assert_close(host(rm), em, "f32", "running mean")
    assert_close(host(rv), ev, "f32", "running var")
    dA = _mat(rng, n, c, dtype)
    dg, db = sscn.batchnorm_relu_backward_params(dev(dA, TD[dtype]), tx, st, dev(b))
    dx = torch.empty_like(tx)
    sscn.batchnorm_relu_backward_input(dev(dA, TD[dtype]), tx, dev(g), dev(b), st, dg, db, dx)
    # the oracle on the same statistics the GPU normalised with
    rdx, rdg, rdb = O.batch_norm_relu_backward(dA, x, g, b, mean, var)
    tol = "f32"   # fp32 outputs of exactly representable inputs
    assert_close(host(dg), rdg, tol, "dgamma")
    assert_close(host(db), rdb, tol, "dbeta")
    assert_close(host(dx), rdx, dtype, "dx")


def test_batchnorm_backward_column_ranges():
    """A concatenation's gradient written as two halves, one with a gradient
    from another consumer added in."""
    rng = np.random.default_rng(5)
    n, c = 5000, 24
    x, dA, other = _mat(rng, n, 2 * c, "f32"), _mat(rng, n, 2 * c, "f32"), _mat(rng, n, c, "f32")
    g = rng.uniform(0.5, 1.5, 2 * c).astype(np.float32)
    b = rng.normal(0, 0.5, 2 * c).astype(np.float32)
    tx, tg, tb = dev(x), dev(g), dev(b)
    st = sscn.batchnorm_forward(tx, tg, tb)
    dg, db = sscn.batchnorm_relu_backward_params(dev(dA), tx, st, tb)
    left, right = torch.empty((n, c), device="cuda:0"), torch.empty((n, c), device="cuda:0")
    sscn.batchnorm_relu_backward_input(dev(dA), tx, tg, tb, st, dg, db, left, add=dev(other), cols=(0, c))
    sscn.batchnorm_relu_backward_input(dev(dA), tx, tg, tb, st, dg, db, right, cols=(c, 2 * c))
    _, mean, var = O.batch_norm_relu_train(x, g, b)
    rdx, _, _ = O.batch_norm_relu_backward(dA, x, g, b, mean, var)
    assert_close(host(left), rdx[:, :c] + other, "f32", "left half + add")
    assert_close(host(right), rdx[:, c:], "f32", "right half")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("n,k", [(1, 2), (3000, 50), (70001, 70)])
def test_softmax_nll(n, k, dtype):
    rng = np.random.default_rng(n + k)
    z = _mat(rng, n, k, dtype, scale=4.0)
    lab = S.labels(n, k, n)
    loss, d = sscn.softmax_nll(dev(z, TD[dtype]), dev(lab))
    rl, rd = O.softmax_nll(z, lab)
    assert abs(float(loss) - rl) <= 1e-5 * abs(rl) + 1e-6
    assert_close(host(d), rd, dtype, "dlogits")


def test_sgd_nesterov_two_steps():
    rng = np.random.default_rng(6)
    p0 = rng.standard_normal(1001).astype(np.float32)
    p, buf = dev(p0.copy()), torch.zeros(1001, device="cuda:0")
    cp = torch.empty(1001, dtype=torch.bfloat16, device="cuda:0")
    rp, rbuf = p0.astype(np.float64), np.zeros(1001)
    for step in range(2):
        g = rng.standard_normal(1001).astype(np.float32)
        sscn.sgd_nesterov_(p, dev(g), buf, 0.1, params_bf16=cp)
        rp, rbuf = O.sgd_nesterov(rp, g, rbuf, 0.1)
        assert_close(host(p), rp, "f32", f"params, step {step}")
        assert_close(host(buf), rbuf, "f32", f"buffer, step {step}")
    np.testing.assert_array_equal(host(cp), S.bf16_round(host(p)))


def test_column_sum_and_add():
    rng = np.random.default_rng(7)
    x = _mat(rng, 30001, 9, "f32")
    assert_close(host(sscn.column_sum(dev(x))), x.astype(np.float64).sum(axis=0), "f32", "column sum")
    y = _mat(rng, 30001, 9, "f32")
    out = torch.empty((30001, 9), device="cuda:0")
    sscn.add_into(dev(x), dev(y), out)
    np.testing.assert_array_equal(host(out), x + y)


def _geometry(batch=2, L=32, per=3000, levels=3):
    coords = S.scenes_small(batch=batch, L=L, target_per_sample=per)
    return coords, (L, L, L)


CH, NCLS = (8, 16, 24), 6


def _draw(name, k, cin, cout):
    return S.train_params(name, k, cin, cout)


def _unit(name):
    if name == "head":
        return unet.Unit("head", "ssc", 0, 1, CH[0], NCLS)
    return {u.name: u for u in unet.units(CH)}[name]


def _input_level(u):
    return u.level + 1 if u.kind == "dc" else (u.level - 1 if u.kind == "sc" else u.level)


def _oracle_levels(coords, size):
    levels, c, sz = [], coords, size
    for l in range(len(CH)):
        ssc = O.ssc_rulebook(c, sz, 3)
        sc = O.sc_rulebook(c, sz, 2, 2) if l + 1 < len(CH) else None
        levels.append((c.shape[0], ssc, sc))
        if sc is not None:
            c, sz = sc.out_coords, sc.out_size
    return levels


def test_train_step_fp32_matches_oracle():
    """One whole step, fp32: loss, every parameter gradient, the running
    statistics and the updated parameters against the oracle's step."""
    coords, size = _geometry()
    n = coords.shape[0]
    X = S.features(n, CH[0], S.SEED_FEAT + 31)
    lab = S.labels(n, NCLS, 32)
    rloss, rgrads, rstats = O.unet_train_step(coords, size, X, lab, _draw, CH, NCLS)
    levels = _oracle_levels(coords, size)
    geom = train.Geometry(dev(coords), size, levels=len(CH))
    P = train.Params(CH, NCLS, _draw)
    loss, grads = train.train_step(dev(X), dev(lab), geom, P)
    assert abs(float(loss) - rloss) <= 1e-5 * abs(rloss)
    assert set(grads) == set(rgrads)
    for name, rg in rgrads.items():
        u = _unit(name)
        for i, (got, want) in enumerate(zip(grads[name], rg)):
            assert_close(host(got).reshape(want.shape), want, "f32", f"{name} grad {i}")
        mean, var = rstats[name]
        em, ev = O.running_stats(np.zeros_like(mean), np.ones_like(var), mean, var, levels[_input_level(u)][0])
        assert_close(host(P.running[name][0]), em, "f32", f"{name} running mean")
        assert_close(host(P.running[name][1]), ev, "f32", f"{name} running var")
        # the update: one Nesterov step from the drawn values (zero momentum buffer)
        for i, (got, p, g) in enumerate(zip(P.master[name], _draw(name, u.k, u.cin, u.cout), rg)):
            want, _ = O.sgd_nesterov(p.astype(np.float64), g.reshape(p.shape), np.zeros(p.shape), 0.1)
            assert_close(host(got), want, "f32", f"{name} param {i} after the step")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_train_step_teacher_forced(dtype):
    """Every unit fed its own GPU tensors (its input x and upstream gradient
    dy) against the oracle's unit: the pre-activation, dA, dW, dgamma, dbeta
    and dx.  dW, dgamma and dbeta are fp32 outputs of exactly representable
    inputs and are held to the fp32 tolerance in both dtypes."""
    coords, size = _geometry()
    n = coords.shape[0]
    X = S.features(n, CH[0], S.SEED_FEAT + 33, bf16=dtype == "bf16")
    lab = S.labels(n, NCLS, 34)
    levels = _oracle_levels(coords, size)
    geom = train.Geometry(dev(coords), size, levels=len(CH))
    P = train.Params(CH, NCLS, _draw, dtype=TD[dtype])
    trace = {}
    _, grads = train.train_step(dev(X, TD[dtype]), dev(lab), geom, P, update=False, trace=trace)
    rnd = O.round_bf16 if dtype == "bf16" else (lambda a: a)
    assert set(trace) == set(grads)
    for name, e in trace.items():
        u = _unit(name)
        if name == "head":
            rb = O.ssc_rulebook(coords, size, 1)
        elif u.kind == "ssc":
            rb = levels[u.level][1]
        elif u.kind == "sc":
            rb = levels[u.level - 1][2]
        else:
            rb = O.transpose(levels[u.level][2])
        p = _draw(name, u.k, u.cin, u.cout)
        g, b = p[0], p[1]
        W = rnd(p[2].astype(np.float64))
        x = host(e["x"])
        A, mean, var = O.batch_norm_relu_train(x, g, b)
        assert_close(host(e["a"]), A, dtype, f"{name} pre-activation")
        da, dW = O.backward(host(e["a"]), W, host(e["dy"]), rb)
        assert_close(host(e["da"]), da, dtype, f"{name} dA")
        assert_close(host(grads[name][2]).reshape(dW.shape), dW, "f32", f"{name} dW")
        dx, dg, db = O.batch_norm_relu_backward(host(e["da"]), x, g, b, mean, var)
        assert_close(host(grads[name][0]), dg, "f32", f"{name} dgamma")
        assert_close(host(grads[name][1]), db, "f32", f"{name} dbeta")
        if name.startswith("down"):       # the skip's gradient joins the one from the SC unit
            dx = dx + host(trace[f"dec{name[4:]}a"]["dx"][0])
        if name == "head":
            assert_close(host(grads[name][3]), host(e["dy"]).astype(np.float64).sum(axis=0), "f32", "head dbias")
        dxs = e["dx"] if isinstance(e["dx"], list) else [e["dx"]]
        assert_close(np.concatenate([host(t) for t in dxs], axis=1), dx, dtype, f"{name} dx")
