"""The C-ABI library loads and exports every symbol include/sscn.h declares.

Also checks the argument validation that happens on the host before any
device work (no GPU needed).
"""
import ctypes

import pytest

from paper_1711_10275_amd import sscn


def test_header_declares_the_boundary():
    names = set(sscn.header_functions())
    for required in ["ssc_rulebook_build", "sc_rulebook_build", "sparse_conv_forward",
                     "sparse_conv_backward", "sscn_rulebook_transpose", "sscn_rulebook_query",
                     "sscn_rulebook_export", "sscn_rulebook_out_coords", "sscn_rulebook_free",
                     "sscn_last_error"]:
        assert required in names


def test_library_exports_every_declared_symbol():
    L = sscn.lib()
    missing = [n for n in sscn.header_functions() if not hasattr(L, n)]
    assert not missing, missing
    assert set(sscn._SIGS) == set(sscn.header_functions())


def _build_ssc(n, size, f, out=True):
    L = sscn.lib()
    h = ctypes.c_void_p()
    sz = (ctypes.c_int32 * 3)(*size)
    return L.ssc_rulebook_build(None, n, sz, f, None, ctypes.byref(h) if out else None)


def test_host_side_validation_codes():
    L = sscn.lib()
    assert _build_ssc(0, (8, 8, 8), 3, out=False) == 1           # NULL out
    assert _build_ssc(-1, (8, 8, 8), 3) == 1                      # n < 0
    assert _build_ssc(5, (8, 8, 8), 3) == 1                       # NULL coords with n > 0
    assert _build_ssc(0, (8, 8, 8), 2) == 1                       # even f for SSC
    assert b"odd" in L.sscn_last_error()
    assert _build_ssc(0, (0, 8, 8), 3) == 1                       # bad extent
    h = ctypes.c_void_p()
    sz = (ctypes.c_int32 * 3)(9, 8, 8)
    assert L.sc_rulebook_build(None, 0, sz, 2, 2, None, ctypes.byref(h)) == 2   # (9-2) % 2 != 0
    sz = (ctypes.c_int32 * 3)(1, 8, 8)
    assert L.sc_rulebook_build(None, 0, sz, 2, 2, None, ctypes.byref(h)) == 2   # L < f
    info = sscn.RulebookInfo()
    assert L.sscn_rulebook_query(None, ctypes.byref(info), None) == 1
    assert L.sparse_conv_forward(None, None, None, 4, 4, 0, None, None) == 1
    L.sscn_rulebook_free(None)  # no-op
    assert L.sscn_affine_relu(None, None, None, 0, 4, 7, None, None) == 1       # bad dtype
    assert L.sscn_concat_cols(None, 4, None, 4, 0, 0, None, None) == 0         # n = 0 is a no-op


def test_binding_refuses_cpu_tensors():
    import torch
    with pytest.raises(ValueError):
        sscn.ssc_rulebook_build(torch.zeros((1, 4), dtype=torch.int32), (8, 8, 8), 3)
