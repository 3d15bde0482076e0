"""Tolerance rule shared by the parity tests.

Per element |y - ref| <= rtol * (|ref| + rms(ref)), rms over the whole
tensor: a relative bound that does not blow up where cancellation makes one
reference element tiny.  fp32: rtol 1e-5; bf16 (products accumulated in
fp32, one rounding to bf16 at the end): rtol 2e-2.  The reference is the
fp64 oracle evaluated on exactly the values the GPU received.
"""
import numpy as np

RTOL = {"f32": 1e-5, "bf16": 2e-2}


def assert_close(got, ref, dtype, what=""):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    if ref.size == 0:
        return
    rms = np.sqrt(np.mean(ref * ref))
    bound = RTOL[dtype] * (np.abs(ref) + rms)
    err = np.abs(got - ref)
    bad = err > bound
    if np.any(bad) or not np.all(np.isfinite(got)):
        i = np.unravel_index(np.argmax(err - bound), err.shape)
        raise AssertionError(f"{what}: {int(bad.sum())} of {bad.size} elements out of tolerance "
                             f"({dtype}); worst at {i}: got {got[i]!r} ref {ref[i]!r} bound {bound[i]:.3g}; "
                             f"normwise {np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-300):.3g}")


def assert_close_head(got, conv_ref, scale, shift, dtype, what=""):
    """An activated output head relu(y * scale + shift) of a convolution
    output y.  The A12 rule bounds y's error by rtol (|y_ref| + rms(y_ref));
    the head multiplies that error by |scale| per channel, and rounding the
    head's own value to the stored dtype adds rtol |head|.  So per element
    |got - relu(y_ref s + t)| <= rtol (|s| (|y_ref| + rms(y_ref)) + |head_ref|).
    (Bounding it by the head value's own magnitude instead fails wherever
    y s nearly cancels t, however accurate y is.)"""
    got = np.asarray(got, np.float64)
    y = np.asarray(conv_ref, np.float64)
    s = np.asarray(scale, np.float64)
    want = np.maximum(0.0, y * s + np.asarray(shift, np.float64))
    assert got.shape == want.shape, (what, got.shape, want.shape)
    if y.size == 0:
        return
    rms = np.sqrt(np.mean(y * y))
    bound = RTOL[dtype] * (np.abs(s) * (np.abs(y) + rms) + np.abs(want))
    err = np.abs(got - want)
    bad = err > bound
    if np.any(bad) or not np.all(np.isfinite(got)):
        i = np.unravel_index(np.argmax(err - bound), err.shape)
        raise AssertionError(f"{what}: {int(bad.sum())} of {bad.size} elements out of tolerance ({dtype}); "
                             f"worst at {i}: got {got[i]!r} ref {want[i]!r} bound {bound[i]:.3g}")
