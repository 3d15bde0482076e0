"""GPU pooling (MP, AP) and nearest-neighbour upsampling, forward and
backward, against the fp64 CPU oracle.  Maxima and copies are exact; sums
are held to the layer tolerances."""
import numpy as np
import pytest
import torch

from oracle import sscn_oracle as O
from paper_1711_10275_amd import sscn
from paper_1711_10275_amd import synthetic as S
from tests.gpu_common import coords_for, dev, host, small_set
from tests.parity import assert_close

pytestmark = pytest.mark.gpu

TD = {"f32": torch.float32, "bf16": torch.bfloat16}
CASES = [((8, 8, 8), 2, 2), ((9, 9, 9), 3, 2), ((9, 9, 9), 3, 3), ((9, 9, 9), 1, 2), ((12, 12, 12), 4, 4)]


def _feat(n, c, seed, dtype):
    return S.features(n, c, seed, bf16=dtype == "bf16")


def _arg(a):
    a = host(a).astype(np.int64)
    return np.where(a == 255, O.NO_ARGMAX, a)


def _check_pool(c, size, f, s, ch, dtype, seed, integer=False):
    rb = sscn.sc_rulebook_build(dev(c), size, f, s)
    orb = O.sc_rulebook(c, size, f, s)
    rng = np.random.default_rng(seed)
    X = rng.integers(-3, 4, (c.shape[0], ch)).astype(np.float32) if integer else _feat(c.shape[0], ch, seed, dtype)
    y, a = sscn.pool_forward(dev(X, TD[dtype]), rb, "max")
    Y, A = O.max_pool(X, orb)
    np.testing.assert_array_equal(host(y), Y)
    np.testing.assert_array_equal(_arg(a), A)
    G = _feat(orb.n_out, ch, seed + 1, dtype)
    dx = sscn.pool_backward(dev(G, TD[dtype]), rb, "max", a)
    assert_close(host(dx), O.max_pool_backward(G, A, orb), dtype, "MP backward")
    ya, _ = sscn.pool_forward(dev(X, TD[dtype]), rb, "avg")
    assert_close(host(ya), O.avg_pool(X, orb), dtype, "AP forward")
    dxa = sscn.pool_backward(dev(G, TD[dtype]), rb, "avg")
    assert_close(host(dxa), O.avg_pool_backward(G, orb), dtype, "AP backward")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("size,f,s", CASES)
def test_pool_small(size, f, s, dtype):
    c = small_set(300 + f * 10 + s, size, batch=2, density=0.3)
    _check_pool(c, size, f, s, 13, dtype, 310 + f)


def test_pool_ties_are_exact():
    """Integer features: many equal maxima; the winning offsets (smallest o)
    and the routed gradients must match exactly."""
    c = small_set(321, (10, 10, 10), batch=2, density=0.6)
    _check_pool(c, (10, 10, 10), 2, 2, 7, "f32", 322, integer=True)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("ch", [64, 70])
def test_pool_shapes128(ch, dtype):
    """The 100k-site surface workload, SC(2, 2) fields, one and two channel chunks."""
    coords, size = coords_for("shapes128")
    _check_pool(coords, size, 2, 2, ch, dtype, 330 + ch)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("config,s", [("small", 2), ("small", 3), ("shapes128", 2)])
def test_upsample(config, s, dtype):
    if config == "small":
        size = (12, 12, 12)
        c = small_set(340 + s, size, batch=2, density=0.3)
    else:
        c, size = coords_for("shapes128")
    rb = sscn.sc_rulebook_build(dev(c), size, s, s)
    orb = O.sc_rulebook(c, size, s, s)
    Y = _feat(orb.n_out, 24, 350 + s, dtype)
    up = sscn.upsample_forward(dev(Y, TD[dtype]), rb)
    np.testing.assert_array_equal(host(up), O.upsample_nearest(Y, orb))
    G = _feat(orb.n_in, 24, 360 + s, dtype)
    dy = sscn.upsample_backward(dev(G, TD[dtype]), rb)
    assert_close(host(dy), O.upsample_nearest_backward(G, orb), dtype, "upsample backward")


def test_pool_argument_errors():
    c = small_set(370, (8, 8, 8), batch=1, density=0.3)
    ssc = sscn.ssc_rulebook_build(dev(c), (8, 8, 8), 3)
    X = torch.zeros((c.shape[0], 4), device="cuda:0")
    with pytest.raises(sscn.SSCNError):
        sscn.pool_forward(X, ssc, "max")
    sc = sscn.sc_rulebook_build(dev(c), (8, 8, 8), 2, 2)
    with pytest.raises(sscn.SSCNError):
        sscn.pool_forward(torch.zeros((sc.n_out, 4), device="cuda:0"), sc.transpose(), "avg")
    sc3 = sscn.sc_rulebook_build(dev(small_set(371, (9, 9, 9), batch=1)), (9, 9, 9), 3, 2)
    with pytest.raises(sscn.SSCNError):
        sscn.upsample_forward(torch.zeros((sc3.n_out, 4), device="cuda:0"), sc3)
