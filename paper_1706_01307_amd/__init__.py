"""Sparse convolutions SC and VSC on MI355X (gfx950).

Python face of libspconv.so.  The functions here marshal torch tensors into
the C ABI (include/spconv.h); all computation runs in the HIP kernels.

    rb = build_rulebook(VSC, coords, spatial_size, f)     # coords: int32 cuda [N, D]
    y  = vsc_forward(rb, x, w, bias)                       # x: [N, C_in], w: [K, C_in, C_out]

A rule book is reusable for every layer with the same site set (Section 4 of
the paper).  Everything runs on torch's current stream.
"""
from __future__ import annotations

import ctypes

import numpy as np

from . import _lib
from ._lib import (BF16, BUILD_ASYNC, BUILD_TRANSPOSE, EDUP, EINVAL, ENOMEM, ERANGE, ECAP,
                   EHIP, F32, OK, OP_DC, OP_SC, OP_VSC, POOL_AVG, POOL_MAX, SC, VSC,
                   SpconvError)

__all__ = ["VSC", "SC", "F32", "BF16", "BUILD_ASYNC", "BUILD_TRANSPOSE", "OP_VSC", "OP_SC",
           "OP_DC", "POOL_MAX", "POOL_AVG", "Rulebook", "build_rulebook", "build_rulebook_on",
           "vsc_forward",
           "sc_forward", "forward_fused", "dc_forward", "pool_forward", "backward_data",
           "backward_weight", "set_allocator", "use_torch_allocator", "release_cached_memory",
           "memory_stats",
           "SpconvError", "OK", "EINVAL", "EDUP", "ERANGE", "ENOMEM", "ECAP", "EHIP"]


def _torch():
    import torch
    return torch


def _stream_ptr(stream=None):
    torch = _torch()
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _dtype_code(t):
    torch = _torch()
    if t == torch.float32:
        return F32
    if t == torch.bfloat16:
        return BF16
    raise TypeError(f"unsupported dtype {t}: use float32 or bfloat16")


def _i32_array(v, D, name):
    a = np.ascontiguousarray(np.asarray(v, dtype=np.int32).reshape(-1))
    if a.size != D:
        raise ValueError(f"{name} needs {D} entries, got {a.size}")
    return a


class Rulebook:
    """Owner of a libspconv rule-book handle."""

    def __init__(self, handle, kind, D, stream):
        self._h = handle
        self.kind = kind
        self.D = D
        self._stream = stream
        self._sizes = None

    @property
    def handle(self):
        return self._h

    def _query(self):
        if self._sizes is None:
            lib = _lib.load()
            n_in, n_out, K = ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int64()
            osz = np.zeros(self.D, np.int32)
            _lib.check(lib.spconv_rulebook_query(self._h, ctypes.byref(n_in), ctypes.byref(n_out),
                                                 ctypes.byref(K), osz.ctypes.data, None),
                       "spconv_rulebook_query")
            off = np.zeros(K.value + 1, np.int64)
            _lib.check(lib.spconv_rulebook_query(self._h, None, None, None, None,
                                                 off.ctypes.data), "spconv_rulebook_query")
            self._sizes = (n_in.value, n_out.value, K.value, osz, off)
        return self._sizes

    def status(self):
        return _lib.load().spconv_rulebook_status(self._h)

    def bounds(self):
        """(input rows, output rows) the buffers are sized for, without waiting."""
        a, b = ctypes.c_int64(), ctypes.c_int64()
        _lib.check(_lib.load().spconv_rulebook_bounds(self._h, ctypes.byref(a), ctypes.byref(b)),
                   "spconv_rulebook_bounds")
        return a.value, b.value

    @property
    def n_in(self):
        return self._query()[0]

    @property
    def n_out(self):
        return self._query()[1]

    @property
    def K(self):
        return self._query()[2]

    @property
    def out_spatial_size(self):
        return self._query()[3].copy()

    @property
    def pair_off(self):
        return self._query()[4].copy()

    def export(self):
        """(out_coords int32 [n_out, D], pairs int32 [sum k, 2]) as cuda tensors."""
        torch = _torch()
        n_out, off = self.n_out, self.pair_off
        oc = torch.empty((n_out, self.D), dtype=torch.int32, device="cuda")
        pr = torch.empty((int(off[-1]), 2), dtype=torch.int32, device="cuda")
        _lib.check(_lib.load().spconv_rulebook_export(
            self._h, oc.data_ptr() if n_out else None, pr.data_ptr() if off[-1] else None,
            _stream_ptr()), "spconv_rulebook_export")
        return oc, pr

    def close(self):
        if self._h:
            _lib.load().spconv_rulebook_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


# ctypes callbacks of every allocator ever registered: a rule book built with
# one calls its release when destroyed, possibly after a later change.
_ALLOCATORS = []


def set_allocator(alloc=None, release=None):
    """Device memory of later rule-book builds from Python callables:
    alloc(nbytes, stream_handle) -> device address (0 = out of memory) and
    release(address, stream_handle).  Both None: back to the library's own
    block cache (see release_cached_memory)."""
    if (alloc is None) != (release is None):
        raise ValueError("give both alloc and release, or neither")
    lib = _lib.load()
    if alloc is None:
        _lib.check(lib.spconv_set_allocator(_lib.ALLOC_FN(), _lib.RELEASE_FN(), None),
                   "spconv_set_allocator")
        return

    def _alloc(nbytes, stream, ctx):
        return int(alloc(int(nbytes), int(stream or 0)) or 0)

    def _release(ptr, stream, ctx):
        release(int(ptr), int(stream or 0))

    pair = (_lib.ALLOC_FN(_alloc), _lib.RELEASE_FN(_release))
    _ALLOCATORS.append(pair)
    _lib.check(lib.spconv_set_allocator(pair[0], pair[1], None), "spconv_set_allocator")


def use_torch_allocator():
    """Rule-book memory from torch's caching allocator (stream-ordered on the
    build stream, like the default)."""
    torch = _torch()

    def alloc(nbytes, stream):
        try:
            return torch.cuda.caching_allocator_alloc(nbytes, torch.cuda.current_device(), stream)
        except RuntimeError:
            return 0

    def release(ptr, stream):
        torch.cuda.caching_allocator_delete(ptr)

    set_allocator(alloc, release)


def release_cached_memory():
    """Free the device memory the library's block cache holds idle (on every
    device); returns the bytes freed.  Rule books alive keep theirs."""
    n = ctypes.c_int64()
    _lib.check(_lib.load().spconv_release_cached_memory(ctypes.byref(n)),
               "spconv_release_cached_memory")
    return n.value


def memory_stats(device=None):
    """(bytes in use, bytes cached idle) of the library's default allocator
    on `device` (default: torch's current device)."""
    torch = _torch()
    dev = torch.cuda.current_device() if device is None else int(device)
    a, b = ctypes.c_int64(), ctypes.c_int64()
    _lib.check(_lib.load().spconv_memory_stats(dev, ctypes.byref(a), ctypes.byref(b)),
               "spconv_memory_stats")
    return a.value, b.value


def build_rulebook(kind, coords, spatial_size, f, s=None, *, sync=True, transpose=False,
                   stream=None):
    """Build the rule book of one SC / VSC layer on the GPU.

    coords: int32 cuda tensor [N, D] (column 0 = sample index).
    spatial_size, f, s: length-D integer sequences, f[0] = s[0] = 1.
    sync=False enqueues the build and returns at once; device-detected
    errors are then reported by Rulebook.status().
    transpose=True (SC only) also builds the reversed pairs that dc_forward
    and the SC input gradient need.
    """
    torch = _torch()
    lib = _lib.load()
    if coords.dtype != torch.int32 or not coords.is_cuda or coords.dim() != 2:
        raise TypeError("coords must be an int32 cuda tensor [N, D]")
    coords = coords.contiguous()
    D = coords.shape[1]
    size = _i32_array(spatial_size, D, "spatial_size")
    fa = _i32_array(f, D, "f")
    sa = _i32_array(np.ones(D) if s is None else s, D, "s")
    h = ctypes.c_void_p()
    st_ptr = _stream_ptr(stream)
    st = lib.spconv_build_rulebook(kind, D, coords.data_ptr() if coords.shape[0] else None,
                                   coords.shape[0], size.ctypes.data, fa.ctypes.data,
                                   sa.ctypes.data,
                                   (0 if sync else BUILD_ASYNC) | (BUILD_TRANSPOSE if transpose else 0),
                                   st_ptr,
                                   ctypes.byref(h))
    _lib.check(st, "spconv_build_rulebook")
    return Rulebook(h, kind, D, st_ptr)


def build_rulebook_on(parent, kind, f, s=None, *, sync=True, stream=None):
    """Rule book of the next layer on the output sites of the SC rule book
    `parent` (its coordinates, grid and device-side count); with sync=False
    nothing waits for the device (see Rulebook.bounds for sizing outputs)."""
    lib = _lib.load()
    if parent.kind != SC:
        raise ValueError("the parent must be an SC rule book")
    D = parent.D
    fa = _i32_array(f, D, "f")
    sa = _i32_array(np.ones(D) if s is None else s, D, "s")
    h = ctypes.c_void_p()
    st_ptr = _stream_ptr(stream)
    _lib.check(lib.spconv_build_rulebook_on(parent.handle, kind, fa.ctypes.data, sa.ctypes.data,
                                            0 if sync else BUILD_ASYNC, st_ptr, ctypes.byref(h)),
               "spconv_build_rulebook_on")
    rb = Rulebook(h, kind, D, st_ptr)
    rb._parent = parent            # its sites are read by the enqueued build
    return rb


def _forward(fn, kind, rb, x, w, bias, out_dtype, out, stream):
    torch = _torch()
    if rb.kind != kind:
        raise ValueError("rule book kind does not match the forward")
    C_in, C_out = int(w.shape[1]), int(w.shape[2])
    in_dt = _dtype_code(x.dtype)
    if w.dtype != x.dtype:
        raise TypeError("x and w must share a dtype")
    out_dtype = x.dtype if out_dtype is None else out_dtype
    out_dt = _dtype_code(out_dtype)
    x = x.contiguous()
    w = w.contiguous()
    if bias is not None:
        bias = bias.contiguous()
        if bias.dtype != torch.float32:
            raise TypeError("bias must be float32")
    if out is None:
        out = torch.empty((rb.n_out, C_out), dtype=out_dtype, device=x.device)
    if out.numel() == 0:
        return out
    st = fn(rb.handle, in_dt, x.data_ptr() if x.numel() else None, w.data_ptr(),
            bias.data_ptr() if bias is not None else None, out_dt,
            out.data_ptr() if out.numel() else None, C_in, C_out, _stream_ptr(stream))
    _lib.check(st, "forward")
    return out


def vsc_forward(rb, x, w, bias=None, out_dtype=None, out=None, stream=None):
    """VSC forward: y[n_out, C_out] = bias + sum_i gathered x @ w[i]."""
    return _forward(_lib.load().spconv_vsc_forward, VSC, rb, x, w, bias, out_dtype, out, stream)


def sc_forward(rb, x, w, bias=None, out_dtype=None, out=None, stream=None):
    """SC forward on an SC rule book (output rows = rb.n_out)."""
    return _forward(_lib.load().spconv_sc_forward, SC, rb, x, w, bias, out_dtype, out, stream)


def forward_fused(rb, x, w, scale=None, shift=None, residual=None, relu=False, out_dtype=None,
                  out=None, stream=None):
    """VSC or SC forward (the book's kind) with the block epilogue fused:
    y = act(acc * scale + shift + residual), scale/shift float32 [C_out] or
    None, residual [n_out, C_out] of the output dtype or None (may be `out`
    itself), act = ReLU if relu."""
    torch = _torch()
    C_in, C_out = int(w.shape[1]), int(w.shape[2])
    if w.dtype != x.dtype:
        raise TypeError("x and w must share a dtype")
    out_dtype = x.dtype if out_dtype is None else out_dtype
    x, w = x.contiguous(), w.contiguous()
    vecs = []
    for v in (scale, shift):
        if v is not None:
            v = v.contiguous()
            if v.dtype != torch.float32:
                raise TypeError("scale and shift must be float32")
        vecs.append(v)
    if out is None:
        out = torch.empty((rb.n_out, C_out), dtype=out_dtype, device=x.device)
    if residual is not None:
        if residual.dtype != out.dtype or tuple(residual.shape) != tuple(out.shape):
            raise TypeError("residual must match the output's dtype and shape")
        if not residual.is_contiguous():
            residual = residual.contiguous()
    if out.numel() == 0:
        return out
    ptr = (lambda t: t.data_ptr() if t is not None else None)
    st = _lib.load().spconv_forward_fused(
        rb.handle, _dtype_code(x.dtype), x.data_ptr() if x.numel() else None, w.data_ptr(),
        ptr(vecs[0]), ptr(vecs[1]), ptr(residual), 1 if relu else 0, _dtype_code(out.dtype),
        out.data_ptr(), C_in, C_out, _stream_ptr(stream))
    _lib.check(st, "spconv_forward_fused")
    return out


def dc_forward(rb, x, w, bias=None, out_dtype=None, out=None, stream=None):
    """Deconvolution DC on the SC rule book it inverts (built with
    transpose=True): x [n_out, C_in] on the SC output sites -> [n_in, C_out]
    on the SC input sites."""
    torch = _torch()
    if rb.kind != SC:
        raise ValueError("DC runs on an SC rule book")
    C_in, C_out = int(w.shape[1]), int(w.shape[2])
    if w.dtype != x.dtype:
        raise TypeError("x and w must share a dtype")
    out_dtype = x.dtype if out_dtype is None else out_dtype
    x, w = x.contiguous(), w.contiguous()
    if bias is not None:
        bias = bias.contiguous()
        if bias.dtype != torch.float32:
            raise TypeError("bias must be float32")
    if out is None:
        out = torch.empty((rb.n_in, C_out), dtype=out_dtype, device=x.device)
    if out.numel() == 0:
        return out
    st = _lib.load().spconv_dc_forward(
        rb.handle, _dtype_code(x.dtype), x.data_ptr() if x.numel() else None, w.data_ptr(),
        bias.data_ptr() if bias is not None else None, _dtype_code(out_dtype), out.data_ptr(),
        C_in, C_out, _stream_ptr(stream))
    _lib.check(st, "spconv_dc_forward")
    return out


def pool_forward(rb, x, mode=POOL_MAX, out=None, stream=None):
    """Sparse MP / AP on an SC rule book: x [n_in, C] -> [n_out, C], same dtype."""
    torch = _torch()
    if rb.kind != SC:
        raise ValueError("pooling runs on an SC rule book")
    x = x.contiguous()
    C = int(x.shape[1])
    if out is None:
        out = torch.empty((rb.n_out, C), dtype=x.dtype, device=x.device)
    if out.numel() == 0:
        return out
    st = _lib.load().spconv_pool_forward(rb.handle, mode, _dtype_code(x.dtype),
                                         x.data_ptr() if x.numel() else None, out.data_ptr(), C,
                                         _stream_ptr(stream))
    _lib.check(st, "spconv_pool_forward")
    return out


def backward_data(rb, op, dy, w, out_dtype=None, out=None, stream=None):
    """Input gradient of a VSC / SC / DC layer (w [K, C_in, C_out] the layer's):
    VSC, SC: dy [n_out, C_out] -> [n_in, C_in]; DC: dy [n_in, C_out] -> [n_out, C_in]."""
    torch = _torch()
    C_in, C_out = int(w.shape[1]), int(w.shape[2])
    if w.dtype != dy.dtype:
        raise TypeError("dy and w must share a dtype")
    out_dtype = dy.dtype if out_dtype is None else out_dtype
    dy, w = dy.contiguous(), w.contiguous()
    rows = rb.n_out if op == OP_DC else rb.n_in
    if out is None:
        out = torch.empty((rows, C_in), dtype=out_dtype, device=dy.device)
    if out.numel() == 0:
        return out
    st = _lib.load().spconv_backward_data(
        rb.handle, op, _dtype_code(dy.dtype), dy.data_ptr() if dy.numel() else None,
        w.data_ptr(), _dtype_code(out_dtype), out.data_ptr(), C_in, C_out, _stream_ptr(stream))
    _lib.check(st, "spconv_backward_data")
    return out


def backward_weight(rb, op, x, dy, C_in, C_out, bias=True, stream=None):
    """(dw float32 [K, C_in, C_out], db float32 [C_out] or None) of a layer."""
    torch = _torch()
    lib = _lib.load()
    if x.dtype != dy.dtype:
        raise TypeError("x and dy must share a dtype")
    x, dy = x.contiguous(), dy.contiguous()
    nbytes = ctypes.c_size_t()
    _lib.check(lib.spconv_backward_weight_workspace(rb.handle, op, C_in, C_out,
                                                     ctypes.byref(nbytes)),
               "spconv_backward_weight_workspace")
    ws = torch.empty(int(nbytes.value), dtype=torch.uint8, device=x.device)
    dw = torch.empty((rb.K, C_in, C_out), dtype=torch.float32, device=x.device)
    db = torch.empty(C_out, dtype=torch.float32, device=x.device) if bias else None
    st = lib.spconv_backward_weight(
        rb.handle, op, _dtype_code(x.dtype), x.data_ptr() if x.numel() else None,
        dy.data_ptr() if dy.numel() else None, dw.data_ptr(),
        db.data_ptr() if db is not None else None, C_in, C_out, ws.data_ptr(), ws.numel(),
        _stream_ptr(stream))
    _lib.check(st, "spconv_backward_weight")
    return dw, db
