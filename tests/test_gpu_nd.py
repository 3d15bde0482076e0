"""Rule books and layers in d = 1, 2 and 4 dimensions on the GPU against the
oracle: bit-exact rule books and output coordinates, then forward, dgrad
and wgrad through the unchanged convolution kernels (K = f^d offsets: the
row-block kernel takes up to 96 of them, with offset sets of one to three
32-bit words: 9, 25, 36 and 49 in d = 2, 16 and 81 in d = 4)."""
import numpy as np
import pytest
import torch

from oracle import sscn_oracle as O
from paper_1711_10275_amd import sscn
from paper_1711_10275_amd import synthetic as S
from tests.gpu_common import assert_same_rulebook, dev, host
from tests.parity import assert_close

pytestmark = pytest.mark.gpu

TD = {"f32": torch.float32, "bf16": torch.bfloat16}


def _set(seed, size, batch=2, density=0.3):
    rng = np.random.default_rng(seed)
    occ = rng.random((batch,) + tuple(size)) < density
    occ[(slice(None),) + (0,) * len(size)] = True
    occ[(slice(None),) + tuple(L - 1 for L in size)] = True
    c = np.argwhere(occ).astype(np.int32)
    return np.ascontiguousarray(c[rng.permutation(c.shape[0])])


CASES = [((40,), 3, 1, True), ((40,), 2, 2, False), ((33, 29), 3, 1, True), ((33, 33), 3, 2, False),
         ((32, 30), 2, 2, False), ((30, 28), 5, 1, True), ((40, 38), 7, 1, True), ((34, 34), 6, 2, False),
         ((9, 8, 7, 9), 3, 1, True), ((8, 8, 6, 6), 2, 2, False), ((9, 9, 9, 7), 3, 2, False)]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("size,f,s,sub", CASES)
def test_nd_layer(size, f, s, sub, dtype):
    c = _set(len(size) * 7 + f * 3 + s, size, density=0.3 if len(size) < 4 else 0.12)
    if sub:
        rb, orb = sscn.ssc_rulebook_build(dev(c), size, f), O.ssc_rulebook(c, size, f)
    else:
        rb, orb = sscn.sc_rulebook_build(dev(c), size, f, s), O.sc_rulebook(c, size, f, s)
    assert rb.dim == len(size) and rb.n_offsets == f ** len(size)
    assert rb.in_size == tuple(size) and rb.out_size == tuple(orb.out_size)
    assert_same_rulebook(rb, orb, f"d={len(size)}")
    np.testing.assert_array_equal(host(rb.out_coords()), orb.out_coords)
    bf = dtype == "bf16"
    for view, oview in ((rb, orb), (rb.transpose(), O.transpose(orb))):
        X = S.features(oview.n_in, 16, 700 + f, bf16=bf)
        W = S.weights(oview.K, 16, 24, 701 + f, bf16=bf)
        y = sscn.sparse_conv_forward(dev(X, TD[dtype]), dev(W, TD[dtype]), view)
        assert_close(host(y), O.forward(X, W, oview), dtype, "forward")
        G = S.features(oview.n_out, 24, 702 + f, bf16=bf)
        dx, dw = sscn.sparse_conv_backward(dev(X, TD[dtype]), dev(W, TD[dtype]), dev(G, TD[dtype]), view)
        rdx, rdw = O.backward(X, W, G, oview)
        assert_close(host(dx), rdx, dtype, "dgrad")
        assert_close(host(dw), rdw, "f32", "wgrad")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_4d_shells_row_blocks(dtype):
    """The 4-d SSC(3) layer of 16 time steps of moving shells (141k sites,
    81 offsets, 2,203 plan blocks of about 70 items): forward and dgrad
    over the row-block plan against the oracle."""
    c = S.moving_shells_4d()
    size = (16, 48, 48, 48)
    rb = sscn.ssc_rulebook_build(dev(c), size, 3)
    orb = O.ssc_rulebook(c, size, 3)
    bf = dtype == "bf16"
    X = S.features(c.shape[0], 32, 710, bf16=bf)
    W = S.weights(81, 32, 32, 711, bf16=bf)
    y = sscn.sparse_conv_forward(dev(X, TD[dtype]), dev(W, TD[dtype]), rb)
    assert_close(host(y), O.forward(X, W, orb), dtype, "4-d forward")
    G = S.features(c.shape[0], 32, 712, bf16=bf)
    dx, _ = sscn.sparse_conv_backward(None, dev(W, TD[dtype]), dev(G, TD[dtype]), rb, wgrad=False)
    assert_close(host(dx), O.backward(X, W, G, orb)[0], dtype, "4-d dgrad")


def test_nd_errors():
    c = dev(_set(1, (8, 8)))
    with pytest.raises(sscn.SSCNError) as e:
        sscn.sc_rulebook_build(c, (9, 8), 2, 2)
    assert e.value.code == "shape"
    bad = _set(2, (8, 8))
    bad[0, 1] = 8
    with pytest.raises(sscn.SSCNError) as e:
        sscn.ssc_rulebook_build(dev(bad), (8, 8), 3)
    assert e.value.code == "out_of_range"
    dup = np.concatenate([_set(3, (8, 8)), _set(3, (8, 8))[:1]])
    with pytest.raises(sscn.SSCNError) as e:
        sscn.ssc_rulebook_build(dev(dup), (8, 8), 3)
    assert e.value.code == "duplicate"
    with pytest.raises(sscn.SSCNError):
        sscn.ssc_rulebook_build(dev(_set(4, (5, 5, 5, 5))), (5, 5, 5, 5), 5)     # 625 offsets
    empty = sscn.ssc_rulebook_build(torch.zeros((0, 3), dtype=torch.int32, device="cuda:0"), (8, 8), 3)
    assert empty.n_pairs == 0 and empty.n_out == 0
    esc = sscn.sc_rulebook_build(torch.zeros((0, 5), dtype=torch.int32, device="cuda:0"), (8, 8, 8, 8), 2, 2)
    assert esc.n_pairs == 0 and esc.n_out == 0
