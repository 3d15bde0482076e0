"""Python binding of libsscn.so (ctypes; argument marshalling only).

Every step of the layers runs in the library's HIP kernels.  torch supplies
device memory (outputs are allocated with torch.empty on the input's device)
and the stream (the current torch stream of that device).  There is no CPU
fallback: if the library is missing or a tensor is not on a GPU, the call
raises.
"""
from __future__ import annotations

import ctypes
import os
import re
import threading

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libsscn.so")
HEADER_PATH = os.path.join(os.path.dirname(_PKG), "include", "sscn.h")

F32, BF16 = 0, 1
STATUS = {0: "ok", 1: "invalid_arg", 2: "shape", 3: "out_of_range", 4: "duplicate", 5: "oom", 6: "device"}
STATUS_CODES = {v: k for k, v in STATUS.items()}


class SSCNError(RuntimeError):
    def __init__(self, code, msg):
        self.code = STATUS.get(code, str(code))
        super().__init__(f"sscn error {self.code}: {msg}")


class RulebookInfo(ctypes.Structure):
    _fields_ = [("n_in", ctypes.c_int64), ("n_out", ctypes.c_int64), ("n_pairs", ctypes.c_int64),
                ("filter_size", ctypes.c_int32), ("stride", ctypes.c_int32),
                ("submanifold", ctypes.c_int32), ("transposed", ctypes.c_int32),
                ("n_offsets", ctypes.c_int32), ("dim", ctypes.c_int32), ("in_size", ctypes.c_int32 * 4),
                ("out_size", ctypes.c_int32 * 4)]


class ConvOutput(ctypes.Structure):
    """sscn_conv_output: one destination of sparse_conv_forward_heads."""
    _fields_ = [("data", ctypes.c_void_p), ("row_stride", ctypes.c_int64), ("scale", ctypes.c_void_p),
                ("shift", ctypes.c_void_p)]


_lib = None
# filter_size is at most 8, so a rule book has at most 8^3 offsets
_MAX_OFFSETS = 512
_vp, _i32, _i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
_SIGS = {
    "ssc_rulebook_build": [_vp, _i64, _vp, _i32, _vp, _vp],
    "sc_rulebook_build": [_vp, _i64, _vp, _i32, _i32, _vp, _vp],
    "sscn_rulebook_build_nd": [_vp, _i64, _i32, _vp, _i32, _i32, _i32, _vp, _vp],
    "sscn_rulebook_transpose": [_vp, _vp],
    "sscn_rulebook_query": [_vp, _vp, _vp],
    "sscn_rulebook_out_coords": [_vp, _vp, _vp],
    "sscn_rulebook_export": [_vp, _vp, _vp, _vp, _vp],
    "sscn_rulebook_free": [_vp],
    "sparse_conv_forward": [_vp, _vp, _vp, _i32, _i32, ctypes.c_int, _vp, _vp],
    "sparse_conv_forward_heads": [_vp, _vp, _vp, _i32, _i32, ctypes.c_int, _i32, _vp, _vp],
    "sparse_conv_forward_noalloc": [_vp, _vp, _vp, _i32, _i32, ctypes.c_int, _vp, _vp],
    "sparse_conv_forward_ex": [_vp, _vp, _vp, _i32, _i32, ctypes.c_int, _vp, _vp, _i64, _i32, _vp, _vp],
    "sparse_conv_backward": [_vp, _vp, _vp, _vp, _i32, _i32, ctypes.c_int, _vp, _vp, _vp],
    "sscn_affine_relu": [_vp, _vp, _vp, _i64, _i32, ctypes.c_int, _vp, _vp],
    "sscn_concat_cols": [_vp, _i32, _vp, _i32, _i64, ctypes.c_int, _vp, _vp],
    "sscn_pool_forward": [_vp, _vp, _i32, ctypes.c_int, ctypes.c_int, _vp, _vp, _vp],
    "sscn_pool_backward": [_vp, _vp, _vp, _i32, ctypes.c_int, ctypes.c_int, _vp, _vp],
    "sscn_upsample_forward": [_vp, _vp, _i32, ctypes.c_int, _vp, _vp],
    "sscn_upsample_backward": [_vp, _vp, _i32, ctypes.c_int, _vp, _vp],
    "sscn_batchnorm_forward": [_vp, _i64, _i64, _i32, ctypes.c_int, _vp, _vp, ctypes.c_float, ctypes.c_float,
                               _vp, _vp, _vp, _vp, _vp, _vp, _vp],
    "sscn_batchnorm_relu_apply": [_vp, _i64, _i64, _i32, ctypes.c_int, _vp, _vp, _vp, _vp, _i64, _vp],
    "sscn_batchnorm_relu_backward_params": [_vp, _i64, _vp, _i64, _i64, _i32, ctypes.c_int, _vp, _vp, _vp, _vp,
                                            _vp, _vp, _vp],
    "sscn_batchnorm_relu_backward_input": [_vp, _i64, _vp, _i64, _i64, _i32, ctypes.c_int, _vp, _vp, _vp, _vp,
                                           _vp, _vp, _vp, _vp, _i64, _vp, _i64, _vp],
    "sscn_column_sum": [_vp, _i64, _i64, _i32, ctypes.c_int, _vp, _vp],
    "sscn_add": [_vp, _i64, _vp, _i64, _i64, _i32, ctypes.c_int, _vp, _i64, _vp],
    "sscn_softmax_nll": [_vp, _i64, _i32, ctypes.c_int, _vp, _vp, _vp, _vp],
    "sscn_sgd_nesterov": [_vp, _vp, _vp, _i64, ctypes.c_float, ctypes.c_float, ctypes.c_float, _vp, _vp],
    "sscn_time_next_launch": [_vp, _vp],
    "sscn_release_cached": [],
    "sscn_set_device_memory_cap": [ctypes.c_uint64],
    "sscn_set_deterministic": [_i32],
    "sscn_last_error": [],
}


def lib():
    """Load libsscn.so (built in-tree by the package's _build module)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it first (__graft_entry__.build())")
        L = ctypes.CDLL(LIB_PATH)
        for name, args in _SIGS.items():
            fn = getattr(L, name)
            fn.argtypes = args
            fn.restype = ctypes.c_char_p if name == "sscn_last_error" else (
                None if name == "sscn_rulebook_free" else ctypes.c_int)
        _lib = L
    return _lib


def header_functions():
    """Names of the functions declared in include/sscn.h."""
    text = open(HEADER_PATH).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(\w+)\s*\([^;{]*\)\s*;", text)) - {"if", "while"})


def _check(code):
    if code != 0:
        raise SSCNError(code, lib().sscn_last_error().decode())


def _stream(t):
    return ctypes.c_void_p(torch.cuda.current_stream(t.device).cuda_stream)


def _dev_tensor(t, name, dtype=None):
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t


def _dtype_code(t):
    if t.dtype == torch.float32:
        return F32
    if t.dtype == torch.bfloat16:
        return BF16
    raise ValueError(f"unsupported dtype {t.dtype} (float32 or bfloat16)")


# per-thread query buffers (a ctypes call releases the GIL while it runs)
_query_bufs = threading.local()


class Rulebook:
    """Owning wrapper of an sscn_rulebook handle."""

    def __init__(self, handle, device):
        self._h = handle
        self.device = device
        bufs = _query_bufs.__dict__
        if not bufs:
            bufs["info"], bufs["ppo"] = RulebookInfo(), (ctypes.c_int64 * _MAX_OFFSETS)()
        info, ppo = bufs["info"], bufs["ppo"]
        _check(lib().sscn_rulebook_query(self._h, ctypes.byref(info), ppo))
        K = info.n_offsets
        self.n_in, self.n_out, self.n_pairs = info.n_in, info.n_out, info.n_pairs
        self.filter_size, self.stride = info.filter_size, info.stride
        self.submanifold, self.transposed = bool(info.submanifold), bool(info.transposed)
        self.n_offsets = K
        self.dim = info.dim
        self.in_size, self.out_size = tuple(info.in_size[:info.dim]), tuple(info.out_size[:info.dim])
        self.pairs_per_offset = list(ppo[:K])

    @property
    def handle(self):
        return self._h

    def transpose(self):
        h = ctypes.c_void_p()
        _check(lib().sscn_rulebook_transpose(self._h, ctypes.byref(h)))
        return Rulebook(h, self.device)

    def out_coords(self):
        out = torch.empty((self.n_out, self.dim + 1), dtype=torch.int32, device=self.device)
        with torch.cuda.device(self.device):
            _check(lib().sscn_rulebook_out_coords(self._h, ctypes.c_void_p(out.data_ptr()), _stream(out)))
        return out

    def export(self):
        """(in_rows, out_rows, offsets) int32 tensors sorted by (offset, out, in)."""
        a = [torch.empty(self.n_pairs, dtype=torch.int32, device=self.device) for _ in range(3)]
        with torch.cuda.device(self.device):
            _check(lib().sscn_rulebook_export(self._h, *[ctypes.c_void_p(x.data_ptr()) for x in a],
                                              _stream(a[0])))
        return tuple(a)

    def macs(self, cin, cout):
        return self.n_pairs * cin * cout

    def free(self):
        if self._h is not None and self._h.value:
            lib().sscn_rulebook_free(self._h)
        self._h = None

    def __del__(self):
        try:
            self.free()
        except Exception:
            pass


_I32x3 = ctypes.c_int32 * 3


def _sizes(spatial_size):
    s = tuple(int(v) for v in spatial_size)
    if len(s) != 3:
        raise ValueError("spatial_size must have 3 entries")
    return _I32x3(*s)


def _build_nd(coords, spatial_size, filter_size, stride, submanifold):
    size = tuple(int(v) for v in spatial_size)
    if not 1 <= len(size) <= 4 or coords.dim() != 2 or coords.shape[1] != len(size) + 1:
        raise ValueError("coords must be n x (d + 1) for d = len(spatial_size) in [1, 4]")
    h = ctypes.c_void_p()
    with torch.cuda.device(coords.device):
        _check(lib().sscn_rulebook_build_nd(ctypes.c_void_p(coords.data_ptr()), coords.shape[0], len(size),
                                            (ctypes.c_int32 * len(size))(*size), int(filter_size), int(stride),
                                            1 if submanifold else 0, _stream(coords), ctypes.byref(h)))
    return Rulebook(h, coords.device)


def ssc_rulebook_build(coords, spatial_size, filter_size=3):
    """SSC rule book; any d = len(spatial_size) in [1, 4] (coords n x (d + 1))."""
    coords = _dev_tensor(coords, "coords", torch.int32)
    if len(spatial_size) != 3:
        return _build_nd(coords, spatial_size, filter_size, 1, True)
    h = ctypes.c_void_p()
    with torch.cuda.device(coords.device):
        _check(lib().ssc_rulebook_build(ctypes.c_void_p(coords.data_ptr()), coords.shape[0],
                                        _sizes(spatial_size), int(filter_size), _stream(coords),
                                        ctypes.byref(h)))
    return Rulebook(h, coords.device)


def sc_rulebook_build(coords, spatial_size, filter_size=2, stride=2):
    """SC rule book; any d = len(spatial_size) in [1, 4] (coords n x (d + 1))."""
    coords = _dev_tensor(coords, "coords", torch.int32)
    if len(spatial_size) != 3:
        return _build_nd(coords, spatial_size, filter_size, stride, False)
    h = ctypes.c_void_p()
    with torch.cuda.device(coords.device):
        _check(lib().sc_rulebook_build(ctypes.c_void_p(coords.data_ptr()), coords.shape[0],
                                       _sizes(spatial_size), int(filter_size), int(stride),
                                       _stream(coords), ctypes.byref(h)))
    return Rulebook(h, coords.device)


def sparse_conv_forward(features, weights, rulebook):
    """out[k] = sum over (j, k) in R_o of features[j] @ weights[o]."""
    features = _dev_tensor(features, "features")
    weights = _dev_tensor(weights, "weights", features.dtype)
    K, cin, cout = weights.shape
    if K != rulebook.n_offsets or features.shape != (rulebook.n_in, cin):
        raise ValueError("features / weights do not match the rule book")
    out = torch.empty((rulebook.n_out, cout), dtype=features.dtype, device=features.device)
    with torch.cuda.device(features.device):
        _check(lib().sparse_conv_forward(ctypes.c_void_p(features.data_ptr()),
                                         ctypes.c_void_p(weights.data_ptr()), rulebook.handle, cin, cout,
                                         _dtype_code(features), ctypes.c_void_p(out.data_ptr()),
                                         _stream(features)))
    return out


def sparse_conv_forward_heads(features, weights, rulebook, heads, bias=None, residual=None):
    """sparse_conv_forward written to 1 or 2 destinations.

    heads: list of (out, scale, shift); out is a device tensor of shape
    (n_out, c_out) in the features' dtype whose rows may be strided (a
    column slice of a wider tensor, unit column stride); scale and shift are
    fp32 (c_out,) device tensors, or None for the plain output.  Each
    destination receives max(0, y * scale + shift), or y.
    """
    features = _dev_tensor(features, "features")
    weights = _dev_tensor(weights, "weights", features.dtype)
    K, cin, cout = weights.shape
    if K != rulebook.n_offsets or features.shape != (rulebook.n_in, cin):
        raise ValueError("features / weights do not match the rule book")
    if not 1 <= len(heads) <= 2:
        raise ValueError("1 or 2 output heads")
    arr = (ConvOutput * len(heads))()
    for i, (out, scale, shift) in enumerate(heads):
        if out.dtype != features.dtype or out.device != features.device or tuple(out.shape) != (rulebook.n_out, cout):
            raise ValueError(f"head {i}: expected a ({rulebook.n_out}, {cout}) {features.dtype} tensor")
        if out.stride(1) != 1:
            raise ValueError(f"head {i}: columns must be contiguous")
        if (scale is None) != (shift is None):
            raise ValueError(f"head {i}: scale and shift go together")
        if scale is not None:
            scale = _dev_tensor(scale, "scale", torch.float32)
            shift = _dev_tensor(shift, "shift", torch.float32)
            if scale.shape != (cout,) or shift.shape != (cout,):
                raise ValueError(f"head {i}: scale / shift must have {cout} entries")
        arr[i].data = out.data_ptr()
        arr[i].row_stride = out.stride(0)
        arr[i].scale = scale.data_ptr() if scale is not None else None
        arr[i].shift = shift.data_ptr() if shift is not None else None
    with torch.cuda.device(features.device):
        if bias is None and residual is None:
            _check(lib().sparse_conv_forward_heads(ctypes.c_void_p(features.data_ptr()),
                                                   ctypes.c_void_p(weights.data_ptr()), rulebook.handle, cin, cout,
                                                   _dtype_code(features), len(heads),
                                                   ctypes.cast(arr, ctypes.c_void_p), _stream(features)))
        else:
            rp, rld = (None, 0)
            if residual is not None:
                rp, rld = _mat(residual, "residual", features.dtype)
                if tuple(residual.shape) != (rulebook.n_out, cout):
                    raise ValueError(f"residual must be ({rulebook.n_out}, {cout})")
            _check(lib().sparse_conv_forward_ex(ctypes.c_void_p(features.data_ptr()),
                                                ctypes.c_void_p(weights.data_ptr()), rulebook.handle, cin, cout,
                                                _dtype_code(features),
                                                _vec(bias, cout, "bias") if bias is not None else None, rp, rld,
                                                len(heads), ctypes.cast(arr, ctypes.c_void_p), _stream(features)))
    return [h[0] for h in heads]


def sparse_conv_forward_ex(features, weights, rulebook, bias=None, residual=None):
    """sparse_conv_forward + bias (per output channel) + residual (n_out x c_out)."""
    out = torch.empty((rulebook.n_out, weights.shape[2]), dtype=features.dtype, device=features.device)
    return sparse_conv_forward_heads(features, weights, rulebook, [(out, None, None)], bias=bias,
                                     residual=residual)[0]


def sparse_conv_backward(features, weights, dout, rulebook, dgrad=True, wgrad=True):
    """(dgrad, wgrad) of sparse_conv_forward; wgrad is float32."""
    weights = _dev_tensor(weights, "weights")
    dout = _dev_tensor(dout, "dout", weights.dtype)
    K, cin, cout = weights.shape
    if K != rulebook.n_offsets or dout.shape != (rulebook.n_out, cout):
        raise ValueError("dout / weights do not match the rule book")
    dev = weights.device
    fptr = None
    if wgrad:
        features = _dev_tensor(features, "features", weights.dtype)
        if features.shape != (rulebook.n_in, cin):
            raise ValueError("features do not match the rule book")
        fptr = ctypes.c_void_p(features.data_ptr())
    dx = torch.empty((rulebook.n_in, cin), dtype=weights.dtype, device=dev) if dgrad else None
    dw = torch.empty((K, cin, cout), dtype=torch.float32, device=dev) if wgrad else None
    with torch.cuda.device(dev):
        _check(lib().sparse_conv_backward(fptr, ctypes.c_void_p(weights.data_ptr()),
                                          ctypes.c_void_p(dout.data_ptr()), rulebook.handle, cin, cout,
                                          _dtype_code(weights),
                                          ctypes.c_void_p(dx.data_ptr()) if dx is not None else None,
                                          ctypes.c_void_p(dw.data_ptr()) if dw is not None else None,
                                          _stream(dout)))
    return dx, dw


POOL_MAX, POOL_AVG = 0, 1


def _vp_of(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else None


def pool_forward(features, rulebook, mode="max"):
    """MP / AP over an SC(f, s) rule book: (out, argmax); argmax (uint8, the
    winning offset per element, 255 for the zero vector) only for "max"."""
    features = _dev_tensor(features, "features")
    n, c = features.shape
    if n != rulebook.n_in:
        raise ValueError("features do not match the rule book")
    m = {"max": POOL_MAX, "avg": POOL_AVG}[mode]
    out = torch.empty((rulebook.n_out, c), dtype=features.dtype, device=features.device)
    arg = torch.empty((rulebook.n_out, c), dtype=torch.uint8, device=features.device) if m == POOL_MAX else None
    with torch.cuda.device(features.device):
        _check(lib().sscn_pool_forward(_vp_of(features), rulebook.handle, c, _dtype_code(features), m,
                                       _vp_of(out), _vp_of(arg), _stream(features)))
    return out, arg


def pool_backward(dout, rulebook, mode="max", argmax=None):
    """Gradient of pool_forward with respect to its features."""
    dout = _dev_tensor(dout, "dout")
    n, c = dout.shape
    if n != rulebook.n_out:
        raise ValueError("dout does not match the rule book")
    m = {"max": POOL_MAX, "avg": POOL_AVG}[mode]
    if m == POOL_MAX:
        argmax = _dev_tensor(argmax, "argmax", torch.uint8)
        if tuple(argmax.shape) != (n, c):
            raise ValueError("argmax must match dout")
    dx = torch.empty((rulebook.n_in, c), dtype=dout.dtype, device=dout.device)
    with torch.cuda.device(dout.device):
        _check(lib().sscn_pool_backward(_vp_of(dout), _vp_of(argmax) if m == POOL_MAX else None, rulebook.handle,
                                        c, _dtype_code(dout), m, _vp_of(dx), _stream(dout)))
    return dx


def upsample_forward(features, rulebook):
    """Nearest-neighbour upsampling back through an SC(s, s) rule book."""
    features = _dev_tensor(features, "features")
    n, c = features.shape
    if n != rulebook.n_out:
        raise ValueError("features must live on the rule book's output sites")
    out = torch.empty((rulebook.n_in, c), dtype=features.dtype, device=features.device)
    with torch.cuda.device(features.device):
        _check(lib().sscn_upsample_forward(_vp_of(features), rulebook.handle, c, _dtype_code(features),
                                           _vp_of(out), _stream(features)))
    return out


def upsample_backward(dout, rulebook):
    dout = _dev_tensor(dout, "dout")
    n, c = dout.shape
    if n != rulebook.n_in:
        raise ValueError("dout must live on the rule book's input sites")
    dy = torch.empty((rulebook.n_out, c), dtype=dout.dtype, device=dout.device)
    with torch.cuda.device(dout.device):
        _check(lib().sscn_upsample_backward(_vp_of(dout), rulebook.handle, c, _dtype_code(dout), _vp_of(dy),
                                            _stream(dout)))
    return dy


def affine_relu(x, scale, shift, out=None):
    """max(0, x * scale + shift) per channel over the active rows."""
    x = _dev_tensor(x, "x")
    n, c = x.shape
    scale = _dev_tensor(scale, "scale", torch.float32)
    shift = _dev_tensor(shift, "shift", torch.float32)
    if scale.numel() != c or shift.numel() != c:
        raise ValueError("scale / shift must have one entry per channel")
    if scale.device != x.device or shift.device != x.device:
        raise ValueError("scale / shift must be on x's device")
    if out is None:
        y = torch.empty_like(x)
    else:
        y = _dev_tensor(out, "out", x.dtype)
        if y.shape != x.shape or y.device != x.device:
            raise ValueError(f"out must be a {tuple(x.shape)} tensor on {x.device}")
    with torch.cuda.device(x.device):
        _check(lib().sscn_affine_relu(ctypes.c_void_p(x.data_ptr()), ctypes.c_void_p(scale.data_ptr()),
                                      ctypes.c_void_p(shift.data_ptr()), n, c, _dtype_code(x),
                                      ctypes.c_void_p(y.data_ptr()), _stream(x)))
    return y


def release_cached(device=None):
    """Return the library's idle device blocks on `device` to the device."""
    with torch.cuda.device(device if device is not None else torch.cuda.current_device()):
        _check(lib().sscn_release_cached())


def set_device_memory_cap(nbytes):
    """Cap the device memory the library holds per device (0: no cap); an
    allocation beyond it fails with the out-of-memory status."""
    _check(lib().sscn_set_device_memory_cap(int(nbytes)))


def set_deterministic(on):
    """wgrad adds its partial sums in a fixed order (bit-reproducible dW)."""
    _check(lib().sscn_set_deterministic(1 if on else 0))


def concat_cols(a, b):
    """[a | b] row by row."""
    a = _dev_tensor(a, "a")
    b = _dev_tensor(b, "b", a.dtype)
    if a.shape[0] != b.shape[0]:
        raise ValueError("row counts differ")
    y = torch.empty((a.shape[0], a.shape[1] + b.shape[1]), dtype=a.dtype, device=a.device)
    with torch.cuda.device(a.device):
        _check(lib().sscn_concat_cols(ctypes.c_void_p(a.data_ptr()), a.shape[1], ctypes.c_void_p(b.data_ptr()),
                                      b.shape[1], a.shape[0], _dtype_code(a), ctypes.c_void_p(y.data_ptr()),
                                      _stream(a)))
    return y


# ---------------------------------------------------------------- training
def _mat(t, name, dtype=None):
    """A row-major matrix view: a 2-D GPU tensor with unit column stride
    (a column slice of a wider tensor is fine).  Returns (pointer, ld)."""
    if not isinstance(t, torch.Tensor) or not t.is_cuda or t.dim() != 2:
        raise ValueError(f"{name} must be a 2-D GPU tensor")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if t.stride(1) != 1 and t.shape[1] > 1:
        raise ValueError(f"{name}: columns must be contiguous")
    return ctypes.c_void_p(t.data_ptr()), max(t.stride(0), t.shape[1])


def _vec(t, c, name):
    t = _dev_tensor(t, name, torch.float32)
    if t.numel() != c:
        raise ValueError(f"{name} must have {c} entries")
    return ctypes.c_void_p(t.data_ptr())


class BatchNormStats:
    """Per-channel results of a batch-statistics normalisation (fp32)."""

    def __init__(self, c, device):
        z = lambda: torch.empty(c, dtype=torch.float32, device=device)
        self.mean, self.invstd, self.scale, self.shift = z(), z(), z(), z()


def batchnorm_forward(x, gamma, beta, eps=1e-5, momentum=0.1, running_mean=None, running_var=None):
    """Batch statistics of x over its rows -> BatchNormStats (mean, invstd,
    scale, shift); updates the running statistics in place if given."""
    xp, ldx = _mat(x, "x")
    n, c = x.shape
    st = BatchNormStats(c, x.device)
    rm = _vec(running_mean, c, "running_mean") if running_mean is not None else None
    rv = _vec(running_var, c, "running_var") if running_var is not None else None
    with torch.cuda.device(x.device):
        _check(lib().sscn_batchnorm_forward(xp, ldx, n, c, _dtype_code(x), _vec(gamma, c, "gamma"),
                                            _vec(beta, c, "beta"), eps, momentum, rm, rv,
                                            _vp_of(st.mean), _vp_of(st.invstd), _vp_of(st.scale),
                                            _vp_of(st.shift), _stream(x)))
    return st


def batchnorm_relu_apply(x, st, beta, out=None):
    """relu((x - mean) * scale + beta) with the statistics of batchnorm_forward."""
    xp, ldx = _mat(x, "x")
    n, c = x.shape
    if out is None:
        out = torch.empty((n, c), dtype=x.dtype, device=x.device)
    op, ldo = _mat(out, "out", x.dtype)
    if tuple(out.shape) != (n, c):
        raise ValueError("out must match x")
    with torch.cuda.device(x.device):
        _check(lib().sscn_batchnorm_relu_apply(xp, ldx, n, c, _dtype_code(x), _vec(st.mean, c, "mean"),
                                               _vec(st.scale, c, "scale"), _vec(beta, c, "beta"), op, ldo,
                                               _stream(x)))
    return out


def batchnorm_relu_backward_params(dA, x, st, beta):
    """(dgamma, dbeta) of batchnorm_relu_apply(x, st, beta) given dA."""
    dp, ldd = _mat(dA, "dA", x.dtype)
    xp, ldx = _mat(x, "x")
    n, c = x.shape
    dg = torch.empty(c, dtype=torch.float32, device=x.device)
    db = torch.empty(c, dtype=torch.float32, device=x.device)
    with torch.cuda.device(x.device):
        _check(lib().sscn_batchnorm_relu_backward_params(dp, ldd, xp, ldx, n, c, _dtype_code(x), _vp_of(st.mean),
                                                         _vp_of(st.invstd), _vp_of(st.scale), _vec(beta, c, "beta"),
                                                         _vp_of(dg), _vp_of(db), _stream(x)))
    return dg, db


def batchnorm_relu_backward_input(dA, x, gamma, beta, st, dgamma, dbeta, out, add=None, cols=None):
    """out = gradient at x (columns `cols` = (lo, hi) of the layer, default
    all) plus `add`; out / add hold just those columns."""
    n, c = x.shape
    lo, hi = cols if cols is not None else (0, c)
    sl = lambda t: t[:, lo:hi]
    v = lambda t: t[lo:hi]
    dp, ldd = _mat(sl(dA), "dA", x.dtype)
    xp, ldx = _mat(sl(x), "x")
    op, ldo = _mat(out, "out", x.dtype)
    if tuple(out.shape) != (n, hi - lo):
        raise ValueError("out must hold the selected columns")
    ap, lda = _mat(add, "add", x.dtype) if add is not None else (None, 0)
    if add is not None and tuple(add.shape) != (n, hi - lo):
        raise ValueError("add must match out")
    k = hi - lo
    with torch.cuda.device(x.device):
        _check(lib().sscn_batchnorm_relu_backward_input(
            dp, ldd, xp, ldx, n, k, _dtype_code(x), _vec(v(gamma), k, "gamma"), _vec(v(beta), k, "beta"),
            _vec(v(st.mean), k, "mean"), _vec(v(st.invstd), k, "invstd"), _vec(v(st.scale), k, "scale"),
            _vec(v(dgamma), k, "dgamma"), _vec(v(dbeta), k, "dbeta"), ap, lda, op, ldo, _stream(x)))
    return out


def column_sum(x):
    xp, ldx = _mat(x, "x")
    n, c = x.shape
    out = torch.empty(c, dtype=torch.float32, device=x.device)
    with torch.cuda.device(x.device):
        _check(lib().sscn_column_sum(xp, ldx, n, c, _dtype_code(x), _vp_of(out), _stream(x)))
    return out


def add_into(a, b, out):
    ap, lda = _mat(a, "a")
    bp, ldb = _mat(b, "b", a.dtype)
    op, ldo = _mat(out, "out", a.dtype)
    n, c = a.shape
    if tuple(b.shape) != (n, c) or tuple(out.shape) != (n, c):
        raise ValueError("shapes differ")
    with torch.cuda.device(a.device):
        _check(lib().sscn_add(ap, lda, bp, ldb, n, c, _dtype_code(a), op, ldo, _stream(a)))
    return out


def softmax_nll(logits, labels):
    """(loss (device fp32 scalar tensor), dlogits)."""
    logits = _dev_tensor(logits, "logits")
    labels = _dev_tensor(labels, "labels", torch.int32)
    n, k = logits.shape
    if labels.shape != (n,):
        raise ValueError("one label per row")
    loss = torch.empty((), dtype=torch.float32, device=logits.device)
    d = torch.empty_like(logits)
    with torch.cuda.device(logits.device):
        _check(lib().sscn_softmax_nll(_vp_of(logits), n, k, _dtype_code(logits), _vp_of(labels), _vp_of(loss),
                                      _vp_of(d), _stream(logits)))
    return loss, d


def sgd_nesterov_(params, grads, buf, lr, momentum=0.9, weight_decay=1e-4, params_bf16=None):
    """In-place Nesterov SGD step on fp32 `params` (contiguous); refreshes
    the bfloat16 copy if given."""
    params = _dev_tensor(params, "params", torch.float32)
    grads = _dev_tensor(grads, "grads", torch.float32)
    buf = _dev_tensor(buf, "momentum buffer", torch.float32)
    if grads.shape != params.shape or buf.shape != params.shape:
        raise ValueError("shapes differ")
    if params_bf16 is not None:
        params_bf16 = _dev_tensor(params_bf16, "params_bf16", torch.bfloat16)
        if params_bf16.shape != params.shape:
            raise ValueError("bf16 copy shape differs")
    with torch.cuda.device(params.device):
        _check(lib().sscn_sgd_nesterov(_vp_of(params), _vp_of(grads), _vp_of(buf), params.numel(), lr, momentum,
                                       weight_decay, _vp_of(params_bf16), _stream(params)))


# ------------------------------------------------------------- measurement
class KernelTimer:
    """HIP events recorded by the library around the next row-block or wgrad
    kernel launched from this thread (sscn_time_next_launch): arm() before
    the call, ms() after synchronising."""

    def __init__(self):
        self._hip = ctypes.CDLL("libamdhip64.so")
        self._hip.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self._hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]
        self._hip.hipEventSynchronize.argtypes = [ctypes.c_void_p]
        self._hip.hipEventDestroy.argtypes = [ctypes.c_void_p]
        self.before, self.after = ctypes.c_void_p(), ctypes.c_void_p()
        for e in (self.before, self.after):
            if self._hip.hipEventCreate(ctypes.byref(e)) != 0:
                raise RuntimeError("hipEventCreate failed")

    def arm(self):
        _check(lib().sscn_time_next_launch(self.before, self.after))

    def ms(self):
        if self._hip.hipEventSynchronize(self.after) != 0:
            raise RuntimeError("hipEventSynchronize failed")
        t = ctypes.c_float()
        if self._hip.hipEventElapsedTime(ctypes.byref(t), self.before, self.after) != 0:
            raise RuntimeError("hipEventElapsedTime failed (was a kernel launched after arm()?)")
        return t.value

    def __del__(self):
        try:
            for e in (self.before, self.after):
                self._hip.hipEventDestroy(e)
        except Exception:
            pass
