"""GPU forward / backward of SSC, SC and DC layers against the fp64 CPU oracle.

wgrad is always checked at the fp32 tolerance: it is an fp32 output, and
with bf16 inputs every product is exact in fp32 (8-bit significands), so
only the fp32 accumulation rounds, as in the fp32 layer."""
import numpy as np
import pytest
import torch

from oracle import sscn_oracle as O
from paper_1711_10275_amd import sscn
from paper_1711_10275_amd import synthetic as S
from tests.gpu_common import coords_for, dev, host, small_set
from tests.parity import assert_close, assert_close_head

pytestmark = pytest.mark.gpu

TD = {"f32": torch.float32, "bf16": torch.bfloat16}


def _draw(n, cin, cout, K, seed, dtype):
    bf = dtype == "bf16"
    X = S.features(n, cin, S.SEED_FEAT + seed, bf16=bf)
    W = S.weights(K, cin, cout, S.SEED_WEIGHT + seed, bf16=bf)
    return X, W


def _fwd(rb, X, W, dtype):
    return host(sscn.sparse_conv_forward(dev(X, TD[dtype]), dev(W, TD[dtype]), rb))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("config,c", [("shell32", 16), ("shapes128", 64)])
def test_ssc_forward_workloads(config, c, dtype):
    coords, size = coords_for(config)
    rb = sscn.ssc_rulebook_build(dev(coords), size, 3)
    orb = O.ssc_rulebook(coords, size, 3)
    X, W = _draw(coords.shape[0], c, c, 27, 1, dtype)
    assert_close(_fwd(rb, X, W, dtype), O.forward(X, W, orb), dtype, f"{config} {dtype}")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_sc_then_ssc_forward(dtype):
    """SC(2,2) 64 -> 96 channels at 128^3 -> 64^3, then SSC 3^3 with 96 channels."""
    coords, size = coords_for("shapes128")
    sc = sscn.sc_rulebook_build(dev(coords), size, 2, 2)
    osc = O.sc_rulebook(coords, size, 2, 2)
    X, W = _draw(coords.shape[0], 64, 96, 8, 2, dtype)
    Y = _fwd(sc, X, W, dtype)
    assert_close(Y, O.forward(X, W, osc), dtype, "sc22")
    oc = host(sc.out_coords())
    ssc = sscn.ssc_rulebook_build(dev(oc), sc.out_size, 3)
    W2 = S.weights(27, 96, 96, S.SEED_WEIGHT + 22, bf16=dtype == "bf16")
    Yr = Y.astype(np.float32)  # the GPU's own SC output feeds both sides
    assert_close(_fwd(ssc, Yr, W2, dtype), O.forward(Yr, W2, O.ssc_rulebook(oc, sc.out_size, 3)), dtype, "ssc64")


CH = [(1, 1), (3, 5), (16, 16), (32, 48), (70, 33), (130, 20), (64, 136), (8, 300), (48, 64), (96, 128)]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("cin,cout", CH)
def test_ssc_forward_channel_shapes(cin, cout, dtype):
    size = (9, 10, 11)
    c = small_set(cin * 7 + cout, size, batch=2, density=0.2)
    rb = sscn.ssc_rulebook_build(dev(c), size, 3)
    X, W = _draw(c.shape[0], cin, cout, 27, cin + cout, dtype)
    assert_close(_fwd(rb, X, W, dtype), O.forward(X, W, O.ssc_rulebook(c, size, 3)), dtype, f"{cin}x{cout}")


@pytest.mark.parametrize("f,s", [(2, 2), (3, 2), (3, 1), (1, 1)])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_sc_and_dc_forward_small(f, s, dtype):
    size = (9, 9, 9) if f == 3 and s == 2 else (8, 8, 8)
    if (f, s) == (1, 1):
        size = (7, 7, 7)
    c = small_set(f * 10 + s, size, batch=2, density=0.25)
    rb = sscn.sc_rulebook_build(dev(c), size, f, s)
    orb = O.sc_rulebook(c, size, f, s)
    X, W = _draw(c.shape[0], 12, 20, f ** 3, 5, dtype)
    assert_close(_fwd(rb, X, W, dtype), O.forward(X, W, orb), dtype, "sc")
    # DC: transposed rule book with its own weights, outputs at the SC input sites
    Xd, Wd = _draw(rb.n_out, 20, 7, f ** 3, 6, dtype)
    assert_close(_fwd(rb.transpose(), Xd, Wd, dtype), O.forward(Xd, Wd, O.transpose(orb)), dtype, "dc")


def test_shapecontext_identity_is_exact():
    """SSC(1,27,3) with identity weights and X[j] = j + 1 decodes the rule book exactly."""
    coords, size = coords_for("shell32")
    n = coords.shape[0]
    rb = sscn.ssc_rulebook_build(dev(coords), size, 3)
    X = (np.arange(n, dtype=np.float32) + 1)[:, None]
    W = np.eye(27, dtype=np.float32).reshape(27, 1, 27)
    Y = _fwd(rb, X, W, "f32")
    orb = O.ssc_rulebook(coords, size, 3)
    np.testing.assert_array_equal(Y, O.forward(X, W, orb))
    for o in range(27):
        k = np.nonzero(Y[:, o])[0]
        np.testing.assert_array_equal(k, orb.outs[o])
        np.testing.assert_array_equal(Y[k, o].astype(np.int64) - 1, orb.ins[o])


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_integer_inputs_are_exact(dtype):
    coords, size = coords_for("shell32")
    rng = np.random.default_rng(0)
    X = rng.integers(-1, 2, (coords.shape[0], 4)).astype(np.float32)
    W = rng.integers(-1, 2, (27, 4, 6)).astype(np.float32)
    rb = sscn.ssc_rulebook_build(dev(coords), size, 3)
    Y = _fwd(rb, X, W, dtype)
    np.testing.assert_array_equal(Y, O.forward(X, W, O.ssc_rulebook(coords, size, 3)))
    G = rng.integers(-1, 2, (coords.shape[0], 6)).astype(np.float32)
    dx, dw = sscn.sparse_conv_backward(dev(X, TD[dtype]), dev(W, TD[dtype]), dev(G, TD[dtype]), rb)
    rdx, rdw = O.backward(X, W, G, O.ssc_rulebook(coords, size, 3))
    np.testing.assert_array_equal(host(dx), rdx)
    np.testing.assert_array_equal(host(dw), rdw)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_ssc_backward_shapes128(dtype):
    """The 128^3 layer (C = 64): dgrad via the transposed rule book and per-offset wgrad."""
    coords, size = coords_for("shapes128")
    rb = sscn.ssc_rulebook_build(dev(coords), size, 3)
    orb = O.ssc_rulebook(coords, size, 3)
    X, W = _draw(coords.shape[0], 64, 64, 27, 4, dtype)
    G = S.features(coords.shape[0], 64, S.SEED_GRAD + 4, bf16=dtype == "bf16")
    dx, dw = sscn.sparse_conv_backward(dev(X, TD[dtype]), dev(W, TD[dtype]), dev(G, TD[dtype]), rb)
    rdx, rdw = O.backward(X, W, G, orb)
    assert_close(host(dx), rdx, dtype, "dgrad")
    assert_close(host(dw), rdw, "f32", "wgrad")
    # dgrad only / wgrad only
    dx2, none = sscn.sparse_conv_backward(None, dev(W, TD[dtype]), dev(G, TD[dtype]), rb, wgrad=False)
    assert none is None
    np.testing.assert_array_equal(host(dx2), host(dx))


@pytest.mark.parametrize("f,s", [(2, 2), (3, 2)])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_sc_and_dc_backward_small(f, s, dtype):
    size = (8, 8, 8) if s == 2 and f == 2 else (9, 9, 9)
    c = small_set(40 + f, size, batch=2, density=0.25)
    rb = sscn.sc_rulebook_build(dev(c), size, f, s)
    orb = O.sc_rulebook(c, size, f, s)
    for view, oview, (cin, cout) in ((rb, orb, (10, 18)), (rb.transpose(), O.transpose(orb), (18, 10))):
        X, W = _draw(view.n_in, cin, cout, f ** 3, 8, dtype)
        G = S.features(view.n_out, cout, S.SEED_GRAD + 8, bf16=dtype == "bf16")
        dx, dw = sscn.sparse_conv_backward(dev(X, TD[dtype]), dev(W, TD[dtype]), dev(G, TD[dtype]), view)
        rdx, rdw = O.backward(X, W, G, oview)
        assert_close(host(dx), rdx, dtype, "dgrad")
        assert_close(host(dw), rdw, "f32", "wgrad")


def test_sc22_backward_shapes128():
    coords, size = coords_for("shapes128")
    rb = sscn.sc_rulebook_build(dev(coords), size, 2, 2)
    orb = O.sc_rulebook(coords, size, 2, 2)
    X, W = _draw(coords.shape[0], 64, 96, 8, 9, "f32")
    G = S.features(rb.n_out, 96, S.SEED_GRAD + 9)
    dx, dw = sscn.sparse_conv_backward(dev(X), dev(W), dev(G), rb)
    rdx, rdw = O.backward(X, W, G, orb)
    assert_close(host(dx), rdx, "f32", "dgrad")
    assert_close(host(dw), rdw, "f32", "wgrad")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("c,cb", [(24, 7), (32, 16), (5, 3)])
def test_affine_relu_and_concat(dtype, c, cb):
    """16-byte chunk paths (rows of whole chunks) and the element paths."""
    rng = np.random.default_rng(3)
    n = 1000
    x = S.bf16_round(rng.standard_normal((n, c)).astype(np.float32)) if dtype == "bf16" else \
        rng.standard_normal((n, c)).astype(np.float32)
    scale = rng.uniform(0.5, 1.5, c).astype(np.float32)
    shift = rng.normal(0, 0.1, c).astype(np.float32)
    y = host(sscn.affine_relu(dev(x, TD[dtype]), dev(scale), dev(shift)))
    ref = np.maximum(0.0, x.astype(np.float64) * scale + shift)
    assert_close(y, ref, dtype, "affine_relu")
    b = rng.standard_normal((n, cb)).astype(np.float32)
    b = S.bf16_round(b) if dtype == "bf16" else b
    cat = host(sscn.concat_cols(dev(x, TD[dtype]), dev(b, TD[dtype])))
    np.testing.assert_array_equal(cat, np.concatenate([x, b], axis=1))


def test_empty_layer():
    empty = torch.zeros((0, 4), dtype=torch.int32, device="cuda:0")
    rb = sscn.ssc_rulebook_build(empty, (8, 8, 8), 3)
    y = sscn.sparse_conv_forward(torch.zeros((0, 4), device="cuda:0"), torch.zeros((27, 4, 5), device="cuda:0"), rb)
    assert y.shape == (0, 5)
    dx, dw = sscn.sparse_conv_backward(torch.zeros((0, 4), device="cuda:0"), torch.zeros((27, 4, 5), device="cuda:0"),
                                       torch.zeros((0, 5), device="cuda:0"), rb)
    assert dx.shape == (0, 4) and float(dw.abs().sum()) == 0.0


def _heads_case(rb, orb, cin, cout, dtype, seed):
    """Two destinations: an activated one (affine + ReLU) written into the
    right half of a wider buffer, and a plain one; both against the oracle's
    convolution followed by the same map, and the buffer's left half must
    stay untouched."""
    rng = np.random.default_rng(seed)
    X, W = _draw(orb.n_in, cin, cout, orb.K, seed, dtype)
    scale = rng.uniform(0.5, 1.5, cout).astype(np.float32)
    shift = rng.normal(0, 0.1, cout).astype(np.float32)
    wide = torch.full((orb.n_out, 2 * cout + 3), 7.0, dtype=TD[dtype], device="cuda:0")
    plain = torch.empty((orb.n_out, cout), dtype=TD[dtype], device="cuda:0")
    sscn.sparse_conv_forward_heads(dev(X, TD[dtype]), dev(W, TD[dtype]), rb,
                                   [(wide[:, cout:2 * cout], dev(scale), dev(shift)), (plain, None, None)])
    ref = O.forward(X, W, orb)
    got = host(wide)
    assert_close_head(got[:, cout:2 * cout], ref, scale, shift, dtype, "activated head")
    assert_close(host(plain), ref, dtype, "plain head")
    assert np.all(got[:, :cout] == 7.0) and np.all(got[:, 2 * cout:] == 7.0), "writes outside the head"


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("cin,cout", [(64, 64), (32, 48), (24, 128)])
def test_forward_heads_ssc(cin, cout, dtype):
    """Activated + plain heads on the 128^3 shapes workload (the row-block
    kernel: 64- and 32-column groups, fp32 with and without the transposed
    weight copy)."""
    coords, size = coords_for("shapes128")
    _heads_case(sscn.ssc_rulebook_build(dev(coords), size, 3), O.ssc_rulebook(coords, size, 3),
                cin, cout, dtype, 41)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("f,cin,cout", [(5, 16, 24), (3, 12, 20), (3, 20, 130)])
def test_forward_heads_fallback_kernels(f, cin, cout, dtype):
    """Heads through the kernels that run where the row-block plan does not:
    125 offsets (5^3 filter: chunk kernels) and input widths that are not a
    multiple of 8 (generic kernel), two heads each."""
    size = (9, 8, 10)
    c = small_set(80 + f + cin, size, batch=2, density=0.2)
    _heads_case(sscn.ssc_rulebook_build(dev(c), size, f), O.ssc_rulebook(c, size, f), cin, cout, dtype, 45 + f)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_forward_heads_sc_and_dc(dtype):
    """Heads on an SC(2, 2) rule book and on its transpose (the DC path)."""
    coords = small_set(29, (20, 18, 22))
    size = (20, 18, 22)
    sc = sscn.sc_rulebook_build(dev(coords), size, 2, 2)
    osc = O.sc_rulebook(coords, size, 2, 2)
    _heads_case(sc, osc, 32, 64, dtype, 43)
    _heads_case(sc.transpose(), O.transpose(osc), 64, 32, dtype, 44)


def test_forward_heads_rejects_bad_heads():
    coords = small_set(30, (6, 6, 6))
    rb = sscn.ssc_rulebook_build(dev(coords), (6, 6, 6), 3)
    X = torch.zeros((coords.shape[0], 4), device="cuda:0")
    W = torch.zeros((27, 4, 8), device="cuda:0")
    out = torch.empty((coords.shape[0], 8), device="cuda:0")
    s = torch.ones(8, device="cuda:0")
    with pytest.raises(ValueError):
        sscn.sparse_conv_forward_heads(X, W, rb, [])
    with pytest.raises(ValueError):
        sscn.sparse_conv_forward_heads(X, W, rb, [(out, s, None)])
    with pytest.raises(ValueError):
        sscn.sparse_conv_forward_heads(X, W, rb, [(out[:, :4], None, None)])
    with pytest.raises(ValueError):
        sscn.sparse_conv_forward_heads(X, W, rb, [(out, None, None)] * 3)


@pytest.mark.parametrize("f,s", [(2, 2), (3, 2), (1, 2), (4, 4), (4, 2)])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_sc_and_dc_row_blocks(f, s, dtype):
    """SC / DC with channel counts the row-block kernel takes (multiples of
    8): forward and backward of both directions.  With f = 1, s = 2 the SC
    inputs at odd positions reach no output, so the DC direction has output
    rows without any pair (they must come out zero).  f = 4 gives 64
    offsets: offset sets of two 32-bit words in both directions' plans."""
    size = (8, 8, 8) if (f, s) in ((2, 2), (4, 4), (4, 2)) else (9, 9, 9)
    c = small_set(60 + 3 * f + s, size, batch=2, density=0.3)
    rb = sscn.sc_rulebook_build(dev(c), size, f, s)
    orb = O.sc_rulebook(c, size, f, s)
    for view, oview, (cin, cout) in ((rb, orb, (16, 24)), (rb.transpose(), O.transpose(orb), (24, 40))):
        X, W = _draw(view.n_in, cin, cout, f ** 3, 9, dtype)
        assert_close(_fwd(view, X, W, dtype), O.forward(X, W, oview), dtype, "forward")
        G = S.features(view.n_out, cout, S.SEED_GRAD + 9, bf16=dtype == "bf16")
        dx, dw = sscn.sparse_conv_backward(dev(X, TD[dtype]), dev(W, TD[dtype]), dev(G, TD[dtype]), view)
        rdx, rdw = O.backward(X, W, G, oview)
        assert_close(host(dx), rdx, dtype, "dgrad")
        assert_close(host(dw), rdw, "f32", "wgrad")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_ssc_filter5(dtype):
    """SSC 5^3 (125 offsets: more than the row-block plan takes, so the
    chunk kernels run) forward and backward."""
    size = (9, 8, 10)
    c = small_set(71, size, batch=2, density=0.2)
    rb = sscn.ssc_rulebook_build(dev(c), size, 5)
    orb = O.ssc_rulebook(c, size, 5)
    X, W = _draw(c.shape[0], 16, 24, 125, 10, dtype)
    assert_close(_fwd(rb, X, W, dtype), O.forward(X, W, orb), dtype, "forward")
    G = S.features(c.shape[0], 24, S.SEED_GRAD + 10, bf16=dtype == "bf16")
    dx, dw = sscn.sparse_conv_backward(dev(X, TD[dtype]), dev(W, TD[dtype]), dev(G, TD[dtype]), rb)
    rdx, rdw = O.backward(X, W, G, orb)
    assert_close(host(dx), rdx, dtype, "dgrad")
    assert_close(host(dw), rdw, "f32", "wgrad")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("c", [16, 32])
def test_packed_items_forward_backward(c, dtype):
    """Short rows in the row kernel: 32 bf16 channels put two items in each
    step, 16 bf16 channels take one item per 64-byte window, and fp32 rows
    of 16 channels one item per 32-channel window of bf16 parts: SSC forward
    and dgrad (the mirror view), SC(2,2) and its transposed (DC) layer,
    against the oracle."""
    coords, size = coords_for("shell32")
    rb = sscn.ssc_rulebook_build(dev(coords), size, 3)
    orb = O.ssc_rulebook(coords, size, 3)
    X, W = _draw(coords.shape[0], c, c, 27, 7 + c, dtype)
    G = S.features(coords.shape[0], c, S.SEED_GRAD + 7 + c, bf16=dtype == "bf16")
    assert_close(_fwd(rb, X, W, dtype), O.forward(X, W, orb), dtype, f"packed ssc {c}")
    dx, _ = sscn.sparse_conv_backward(None, dev(W, TD[dtype]), dev(G, TD[dtype]), rb, wgrad=False)
    assert_close(host(dx), O.backward(X, W, G, orb)[0], dtype, f"packed dgrad {c}")
    sc = sscn.sc_rulebook_build(dev(coords), size, 2, 2)
    osc = O.sc_rulebook(coords, size, 2, 2)
    Xs, Ws = _draw(coords.shape[0], c, 2 * c, 8, 9 + c, dtype)
    Y = _fwd(sc, Xs, Ws, dtype)
    assert_close(Y, O.forward(Xs, Ws, osc), dtype, f"packed sc {c}")
    Yd, Wd = _draw(sc.n_out, c, c, 8, 11 + c, dtype)
    assert_close(_fwd(sc.transpose(), Yd, Wd, dtype), O.forward(Yd, Wd, O.transpose(osc)), dtype, f"packed dc {c}")


@pytest.mark.parametrize("dtype,c", [("f32", 16), ("f32", 64), ("bf16", 16), ("bf16", 32), ("bf16", 64)])
def test_forward_dgrad_independent_of_row_order(dtype, c):
    """A row's forward and dgrad result is a sum over its own neighbours in
    ascending offset order, whichever rows share its block of the plan: the
    same sites listed in another order give bit-identical rows."""
    coords, size = coords_for("shapes128")
    n = coords.shape[0]
    perm = np.random.default_rng(S.SEED_GEOM + 77).permutation(n)
    X, W = _draw(n, c, c, 27, 60 + c, dtype)
    G = S.features(n, c, S.SEED_GRAD + 60 + c, bf16=dtype == "bf16")
    outs = []
    for order in (np.arange(n), perm):
        rb = sscn.ssc_rulebook_build(dev(np.ascontiguousarray(coords[order])), size, 3)
        y = _fwd(rb, X[order], W, dtype)
        dx, _ = sscn.sparse_conv_backward(None, dev(W, TD[dtype]), dev(G[order], TD[dtype]), rb, wgrad=False)
        outs.append((y, host(dx)))
    np.testing.assert_array_equal(outs[1][0], outs[0][0][perm])
    np.testing.assert_array_equal(outs[1][1], outs[0][1][perm])


WG_ROWS = [("shell32", 32, 32), ("shell32", 64, 32), ("shell32", 64, 64), ("shell32", 128, 64),
           ("shell32", 96, 160), ("shapes128", 32, 32), ("shapes128", 64, 32), ("shapes128", 64, 64),
           ("shapes128", 128, 64), ("shapes128", 96, 64), ("shapes128", 128, 32), ("shapes128", 96, 96),
           ("shapes128", 192, 96), ("shapes128", 128, 128), ("shapes128", 256, 128), ("shapes128", 96, 128),
           ("shapes128", 160, 160), ("shapes128", 128, 160)]


@pytest.mark.parametrize("config,cin,cout", WG_ROWS)
def test_wgrad_row_blocks_bf16(config, cin, cout):
    """bf16 wgrad runs over the row-block plan (gathered rows into LDS,
    transposed operand reads, partial sums added in a fixed order) for
    32 to 160 output channels, with the input channels in one tile or split
    into tiles of 32 or 64: SSC and its mirror view at the fp32 tolerance
    against the oracle, bit-identical on a second call, and the same from a
    wgrad-only call."""
    coords, size = coords_for(config)
    rb = sscn.ssc_rulebook_build(dev(coords), size, 3)
    orb = O.ssc_rulebook(coords, size, 3)
    n = coords.shape[0]
    X, W = _draw(n, cin, cout, 27, 20 + cin + cout, "bf16")
    G = S.features(n, cout, S.SEED_GRAD + 20 + cin + cout, bf16=True)
    for view, oview in ((rb, orb), (rb.transpose(), O.transpose(orb))):
        dx, dw = sscn.sparse_conv_backward(dev(X, torch.bfloat16), dev(W, torch.bfloat16),
                                           dev(G, torch.bfloat16), view)
        rdw = O.backward(X, W, G, oview)[1]
        assert_close(host(dw), rdw, "f32", f"row-block wgrad {config} {cin}x{cout}")
        _, dw2 = sscn.sparse_conv_backward(dev(X, torch.bfloat16), dev(W, torch.bfloat16),
                                           dev(G, torch.bfloat16), view, dgrad=False)
        np.testing.assert_array_equal(host(dw2), host(dw))


@pytest.mark.parametrize("cin,cout", [(32, 32), (64, 32), (96, 128), (160, 128)])
def test_wgrad_row_blocks_sc_dc_bf16(cin, cout):
    """The row-block bf16 wgrad on SC(2,2) (8 offsets) and on its transposed
    (DC) layer, whose plan is built on first use."""
    coords, size = coords_for("shell32")
    sc = sscn.sc_rulebook_build(dev(coords), size, 2, 2)
    osc = O.sc_rulebook(coords, size, 2, 2)
    for view, oview in ((sc, osc), (sc.transpose(), O.transpose(osc))):
        X, W = _draw(view.n_in, cin, cout, 8, 30 + cin, "bf16")
        G = S.features(view.n_out, cout, S.SEED_GRAD + 30 + cin, bf16=True)
        dx, dw = sscn.sparse_conv_backward(dev(X, torch.bfloat16), dev(W, torch.bfloat16),
                                           dev(G, torch.bfloat16), view)
        rdx, rdw = O.backward(X, W, G, oview)
        assert_close(host(dx), rdx, "bf16", f"dgrad sc/dc {cin}")
        assert_close(host(dw), rdw, "f32", f"row-block wgrad sc/dc {cin}")


@pytest.mark.parametrize("dtype,cin,cout", [("f32", 64, 64), ("bf16", 48, 80)])
def test_wgrad_deterministic_mode(dtype, cin, cout):
    """With the deterministic mode the per-pair wgrad writes each work item's
    block to its own slot and adds them in a fixed order: two runs give
    bit-identical dW, which matches the oracle at the fp32 tolerance (and
    the atomic mode's result likewise), on the layer and its mirror view."""
    coords, size = coords_for("shapes128")
    rb = sscn.ssc_rulebook_build(dev(coords), size, 3)
    orb = O.ssc_rulebook(coords, size, 3)
    n = coords.shape[0]
    X, W = _draw(n, cin, cout, 27, 50 + cin, dtype)
    G = S.features(n, cout, S.SEED_GRAD + 50 + cin, bf16=dtype == "bf16")
    for view, oview in ((rb, orb), (rb.transpose(), O.transpose(orb))):
        rdw = O.backward(X, W, G, oview)[1]
        args = (dev(X, TD[dtype]), dev(W, TD[dtype]), dev(G, TD[dtype]), view)
        try:
            sscn.set_deterministic(True)
            _, d1 = sscn.sparse_conv_backward(*args, dgrad=False)
            _, d2 = sscn.sparse_conv_backward(*args)
        finally:
            sscn.set_deterministic(False)
        np.testing.assert_array_equal(host(d1), host(d2))
        assert_close(host(d1), rdw, "f32", "deterministic wgrad")
        _, da = sscn.sparse_conv_backward(*args, dgrad=False)
        assert_close(host(da), rdw, "f32", "atomic wgrad")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("cin,cout", [(32, 20), (20, 32), (64, 64), (8, 300), (3, 5), (70, 33)])
def test_filter1_per_row(cin, cout, dtype):
    """SSC of filter size 1 (one offset, every row paired with itself: a
    per-row linear map), on the row-block and the generic kernels: forward
    with and without a bias, dgrad and wgrad against the oracle."""
    coords, size = coords_for("shapes128")
    rb = sscn.ssc_rulebook_build(dev(coords), size, 1)
    orb = O.ssc_rulebook(coords, size, 1)
    n = coords.shape[0]
    X, W = _draw(n, cin, cout, 1, 80 + cin, dtype)
    assert_close(_fwd(rb, X, W, dtype), O.forward(X, W, orb), dtype, f"f=1 forward {cin}x{cout}")
    bias = S.features(1, cout, S.SEED_WEIGHT + 81 + cin)[0]
    y = sscn.sparse_conv_forward_ex(dev(X, TD[dtype]), dev(W, TD[dtype]), rb, bias=dev(bias, torch.float32))
    assert_close(host(y), O.forward_bias(X, W, bias, orb), dtype, f"f=1 bias {cin}x{cout}")
    G = S.features(n, cout, S.SEED_GRAD + 82 + cin, bf16=dtype == "bf16")
    dx, dw = sscn.sparse_conv_backward(dev(X, TD[dtype]), dev(W, TD[dtype]), dev(G, TD[dtype]), rb)
    rdx, rdw = O.backward(X, W, G, orb)
    assert_close(host(dx), rdx, dtype, f"f=1 dgrad {cin}x{cout}")
    assert_close(host(dw), rdw, "f32", f"f=1 wgrad {cin}x{cout}")
