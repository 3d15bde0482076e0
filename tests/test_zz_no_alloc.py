"""The no-allocation forward (sparse_conv_forward_noalloc), called through the
C ABI, against sparse_conv_forward on the same inputs: the same kernels run,
so the outputs must be bit-identical.  Two calls in a row share the scratch
region, the second with a smaller input; then the error paths (weights too
large for the region, a rule book whose tables are not built yet)."""
import ctypes

import numpy as np
import pytest
import torch

from paper_1711_10275_amd import sscn
from paper_1711_10275_amd import synthetic as S
from tests.gpu_common import coords_for, dev, small_set

pytestmark = pytest.mark.gpu

TD = {"f32": torch.float32, "bf16": torch.bfloat16}


def _noalloc(X, W, rb, out):
    K, cin, cout = W.shape
    code = sscn.F32 if X.dtype == torch.float32 else sscn.BF16
    stream = ctypes.c_void_p(torch.cuda.current_stream(X.device).cuda_stream)
    return sscn.lib().sparse_conv_forward_noalloc(ctypes.c_void_p(X.data_ptr()), ctypes.c_void_p(W.data_ptr()),
                                                  rb.handle, cin, cout, code, ctypes.c_void_p(out.data_ptr()), stream)


def _case(coords, size, cin, cout, dtype, seed, kind="ssc"):
    rb = sscn.ssc_rulebook_build(dev(coords), size, 3) if kind == "ssc" else sscn.sc_rulebook_build(dev(coords), size, 2, 2)
    X = dev(S.features(rb.n_in, cin, seed, bf16=dtype == "bf16"), TD[dtype])
    W = dev(S.weights(rb.n_offsets, cin, cout, seed + 1, bf16=dtype == "bf16"), TD[dtype])
    ref = sscn.sparse_conv_forward(X, W, rb)        # also builds any table the rule book lacks
    return rb, X, W, ref


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_noalloc_matches_forward_twice(dtype):
    big = _case(*coords_for("shapes128"), 64, 64, dtype, 2101)       # 100k sites, 64 -> 64
    small = _case(*coords_for("shell32"), 16, 24, dtype, 2103)        # 1.8k sites, 16 -> 24
    for rb, X, W, ref in (big, small):
        out = torch.full_like(ref, float("nan"))
        assert _noalloc(X, W, rb, out) == 0, sscn.lib().sscn_last_error().decode()
        torch.cuda.synchronize()
        assert torch.equal(out, ref)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_noalloc_other_kernels_twice(dtype):
    """Channel counts the row-block kernel does not take (generic kernel), an
    SC rule book and its transpose, then a smaller SSC layer."""
    c = small_set(501, (12, 12, 12), batch=2, density=0.2)
    cases = [_case(c, (12, 12, 12), 12, 20, dtype, 2105),
             _case(c, (12, 12, 12), 32, 48, dtype, 2107, kind="sc"),
             _case(c[: c.shape[0] // 3], (12, 12, 12), 12, 8, dtype, 2109)]
    sc = cases[1][0]
    Xt = dev(S.features(sc.n_out, 48, 2111, bf16=dtype == "bf16"), TD[dtype])
    Wt = dev(S.weights(8, 48, 32, 2112, bf16=dtype == "bf16"), TD[dtype])
    dc = sc.transpose()
    cases.insert(2, (dc, Xt, Wt, sscn.sparse_conv_forward(Xt, Wt, dc)))
    for rb, X, W, ref in cases:
        out = torch.full_like(ref, float("nan"))
        assert _noalloc(X, W, rb, out) == 0, sscn.lib().sscn_last_error().decode()
        torch.cuda.synchronize()
        assert torch.equal(out, ref)


def test_noalloc_errors():
    c = small_set(503, (8, 8, 8), batch=1, density=0.2)
    rb = sscn.ssc_rulebook_build(dev(c), (8, 8, 8), 3)
    X = torch.zeros((rb.n_in, 512), device="cuda:0")
    W = torch.zeros((27, 512, 256), device="cuda:0")     # 14 MiB of fp32 weights
    out = torch.full((rb.n_out, 256), 3.0, device="cuda:0")
    assert _noalloc(X, W, rb, out) == sscn.STATUS_CODES["invalid_arg"]
    assert "scratch" in sscn.lib().sscn_last_error().decode()
    # an SC rule book builds its tables on first use: not allowed here
    sc = sscn.sc_rulebook_build(dev(c), (8, 8, 8), 2, 2)
    Xs = torch.ones((sc.n_in, 16), device="cuda:0")
    Ws = torch.ones((8, 16, 16), device="cuda:0")
    outs = torch.full((sc.n_out, 16), 3.0, device="cuda:0")
    assert _noalloc(Xs, Ws, sc, outs) == sscn.STATUS_CODES["invalid_arg"]
    assert "not built" in sscn.lib().sscn_last_error().decode()
    torch.cuda.synchronize()
    assert bool((out == 3.0).all()) and bool((outs == 3.0).all())
