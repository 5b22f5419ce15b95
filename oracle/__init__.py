"""Oracle for SC / VSC (TEST INFRASTRUCTURE ONLY).

A ctypes wrapper around ``oracle.cpp``, the plain std::map CPU statement of
the paper's sparse convolutions (Section 3 for the layer definitions,
including sparse max / average pooling and the deconvolution DC, Section 4
for the rule book and the forward multiply-add), plus the derivatives of
those sums that training needs (input, weight and bias gradients), and the
per-channel affine / residual / ReLU epilogue of Section 5's blocks.  Only the test
suite, the smoke check and the benchmark's CPU-baseline leg import this
package; the product path never does.  It shares no code with the HIP
library.

Parity pins for every function here live in ``tests/test_oracle_pins.py``
and ``tests/test_oracle_pins_ext.py``.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.cpp")
_LIB = os.path.join(_HERE, "liboracle.so")

OK, EINVAL, EDUP, ERANGE = 0, -1, -2, -3
VSC, SC, DC = 0, 1, 2
POOL_MAX, POOL_AVG = 0, 1
F32, BF16 = 0, 1


def build():
    """Compile oracle.cpp into liboracle.so (plain g++, host code only; its
    loops over output rows run on OpenMP threads)."""
    cmd = ["g++", "-O2", "-std=c++17", "-fopenmp", "-shared", "-fPIC", "-o", _LIB + ".tmp",
           _SRC]
    subprocess.run(cmd, check=True)
    os.replace(_LIB + ".tmp", _LIB)


_lib = None


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        build()
    lib = ctypes.CDLL(_LIB)
    P, I64, I32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int
    lib.ref_build.argtypes = [I32, I32, P, I64, P, P, P, ctypes.POINTER(P)]
    lib.ref_build.restype = I32
    lib.ref_query.argtypes = [P, P, P, P, P, P]
    lib.ref_query.restype = I32
    lib.ref_export.argtypes = [P, P, P]
    lib.ref_export.restype = I32
    lib.ref_forward.argtypes = [P, I32, P, P, P, I32, I32, P, P, P]
    lib.ref_forward.restype = I32
    lib.ref_forward_rows.argtypes = [P, I32, P, P, P, I32, I32, P, P, P]
    lib.ref_forward_rows.restype = I32
    lib.ref_pool.argtypes = [P, I32, I32, P, I32, P, P]
    lib.ref_pool.restype = I32
    lib.ref_dc_forward.argtypes = [P, I32, P, P, P, I32, I32, P, P, P]
    lib.ref_dc_forward.restype = I32
    lib.ref_backward_data.argtypes = [P, I32, I32, P, P, I32, I32, P, P]
    lib.ref_backward_data.restype = I32
    lib.ref_backward_weight.argtypes = [P, I32, I32, P, P, I32, I32, P, P, P, P, P]
    lib.ref_backward_weight.restype = I32
    lib.ref_round.argtypes = [P, I64, I32, P]
    lib.ref_round.restype = I32
    lib.ref_free.argtypes = [P]
    lib.ref_free.restype = None
    lib.ref_set_threads.argtypes = [I32]
    lib.ref_set_threads.restype = I32
    _lib = lib
    return lib


def set_threads(n):
    """Threads for the oracle's parallel loops (n <= 0 keeps the current
    setting); returns the count in effect.  Results do not depend on it."""
    return int(_load().ref_set_threads(int(n)))


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


class OracleError(RuntimeError):
    def __init__(self, status):
        super().__init__(f"oracle status {status}")
        self.status = status


class Rulebook:
    """Rule book of one SC/VSC layer as computed by the oracle."""

    def __init__(self, kind, coords, spatial_size, f, s=None):
        lib = _load()
        coords = np.ascontiguousarray(coords, dtype=np.int32)
        D = coords.shape[1]
        self.D = D
        size = np.ascontiguousarray(spatial_size, dtype=np.int32)
        f = np.ascontiguousarray(f, dtype=np.int32)
        s = np.ones(D, np.int32) if s is None else np.ascontiguousarray(s, dtype=np.int32)
        h = ctypes.c_void_p()
        st = lib.ref_build(kind, D, _ptr(coords), coords.shape[0], _ptr(size),
                           _ptr(f), _ptr(s), ctypes.byref(h))
        if st != OK:
            raise OracleError(st)
        self._h = h
        n_in, n_out, K = ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int64()
        lib.ref_query(h, ctypes.byref(n_in), ctypes.byref(n_out),
                      ctypes.byref(K), None, None)
        self.n_in, self.n_out, self.K = n_in.value, n_out.value, K.value
        self.out_size = np.zeros(D, np.int32)
        self.pair_off = np.zeros(self.K + 1, np.int64)
        lib.ref_query(h, None, None, None, _ptr(self.out_size), _ptr(self.pair_off))
        self.out_coords = np.zeros((self.n_out, D), np.int32)
        self.pairs = np.zeros((int(self.pair_off[-1]), 2), np.int32)
        lib.ref_export(h, _ptr(self.out_coords), _ptr(self.pairs))

    def offset_pairs(self, i):
        return self.pairs[self.pair_off[i]:self.pair_off[i + 1]]

    def forward(self, x, w, bias=None, in_dt=F32, x_absb=None):
        """Exact-as-double output and absolute-sum bound, both [n_out, C_out].

        x: [n_in, C_in] float32 (in_dt F32) or uint16 bf16 bits (BF16);
        w: [K, C_in, C_out] same dtype; bias: float32 [C_out] or None.
        """
        lib = _load()
        x = np.ascontiguousarray(x)
        w = np.ascontiguousarray(w)
        C_in, C_out = w.shape[1], w.shape[2]
        y = np.zeros((self.n_out, C_out), np.float64)
        absb = np.zeros((self.n_out, C_out), np.float64)
        b = None if bias is None else np.ascontiguousarray(bias, dtype=np.float32)
        xa = None if x_absb is None else np.ascontiguousarray(x_absb, dtype=np.float64)
        st = lib.ref_forward(self._h, in_dt, _ptr(x), _ptr(w), _ptr(b), C_in,
                             C_out, _ptr(y), _ptr(absb), _ptr(xa))
        if st != OK:
            raise OracleError(st)
        return y, absb

    def forward_rows(self, rows, x, w, bias=None, in_dt=F32):
        """Output rows `rows` only: (y [len(rows), C_out], absb) in float64."""
        lib = _load()
        x = np.ascontiguousarray(x)
        w = np.ascontiguousarray(w)
        C_in, C_out = w.shape[1], w.shape[2]
        mask = np.zeros(self.n_out, np.uint8)
        mask[np.asarray(rows)] = 1
        y = np.zeros((self.n_out, C_out), np.float64)
        absb = np.zeros((self.n_out, C_out), np.float64)
        b = None if bias is None else np.ascontiguousarray(bias, dtype=np.float32)
        st = lib.ref_forward_rows(self._h, in_dt, _ptr(x), _ptr(w), _ptr(b), C_in, C_out,
                                  _ptr(mask), _ptr(y), _ptr(absb))
        if st != OK:
            raise OracleError(st)
        return y[rows], absb[rows]

    def pool(self, x, mode, dt=F32):
        """Sparse MP / AP (SC rule book): (y, absb), float64 [n_out, C]."""
        lib = _load()
        x = np.ascontiguousarray(x)
        C = x.shape[1]
        y = np.zeros((self.n_out, C), np.float64)
        absb = np.zeros((self.n_out, C), np.float64)
        st = lib.ref_pool(self._h, mode, dt, _ptr(x), C, _ptr(y), _ptr(absb))
        if st != OK:
            raise OracleError(st)
        return y, absb

    def dc_forward(self, x, w, bias=None, in_dt=F32, x_absb=None):
        """DC on this SC rule book: x [n_out, C_in] -> (y, absb) [n_in, C_out]."""
        lib = _load()
        x = np.ascontiguousarray(x)
        w = np.ascontiguousarray(w)
        C_in, C_out = w.shape[1], w.shape[2]
        y = np.zeros((self.n_in, C_out), np.float64)
        absb = np.zeros((self.n_in, C_out), np.float64)
        b = None if bias is None else np.ascontiguousarray(bias, dtype=np.float32)
        xa = None if x_absb is None else np.ascontiguousarray(x_absb, dtype=np.float64)
        st = lib.ref_dc_forward(self._h, in_dt, _ptr(x), _ptr(w), _ptr(b), C_in, C_out,
                                _ptr(y), _ptr(absb), _ptr(xa))
        if st != OK:
            raise OracleError(st)
        return y, absb

    def backward_data(self, op, dy, w, dt=F32):
        """Input gradient of op (VSC, SC or DC) given dy: (dx, absb) float64."""
        lib = _load()
        dy = np.ascontiguousarray(dy)
        w = np.ascontiguousarray(w)
        C_in, C_out = w.shape[1], w.shape[2]
        rows = self.n_out if op == DC else self.n_in
        dx = np.zeros((rows, C_in), np.float64)
        absb = np.zeros((rows, C_in), np.float64)
        st = lib.ref_backward_data(self._h, op, dt, _ptr(dy), _ptr(w), C_in, C_out,
                                   _ptr(dx), _ptr(absb))
        if st != OK:
            raise OracleError(st)
        return dx, absb

    def backward_weight(self, op, x, dy, C_in, C_out, dt=F32, offsets=None):
        """(dw [K, C_in, C_out], db [C_out], absb_w, absb_b), all float64.

        offsets: indices of the W^i to compute (the others stay zero), or
        None for all of them."""
        lib = _load()
        x = np.ascontiguousarray(x)
        dy = np.ascontiguousarray(dy)
        dw = np.zeros((self.K, C_in, C_out), np.float64)
        aw = np.zeros_like(dw)
        db = np.zeros(C_out, np.float64)
        ab = np.zeros(C_out, np.float64)
        mask = None
        if offsets is not None:
            mask = np.zeros(self.K, np.uint8)
            mask[np.asarray(offsets)] = 1
        st = lib.ref_backward_weight(self._h, op, dt, _ptr(x), _ptr(dy), C_in, C_out,
                                     _ptr(dw), _ptr(db), _ptr(aw), _ptr(ab), _ptr(mask))
        if st != OK:
            raise OracleError(st)
        return dw, db, aw, ab

    def __del__(self):
        h = getattr(self, "_h", None)
        if h is not None and _lib is not None:
            _lib.ref_free(h)
            self._h = None


def fused_epilogue(y, absb, scale=None, shift=None, residual=None, relu=False, res_dt=F32):
    """Per-channel affine map, residual add and ReLU on an exact layer output.

    The networks of Section 5 follow their sparse convolutions with batch
    normalisation and a ReLU, both acting on the active sites only, and their
    residual blocks add the block input back before the last ReLU.  At
    inference a batch normalisation is an affine map per channel, so for an
    output row r and channel n (y and absb from ``forward``):

        z = y[r, n] * scale[n] + shift[n] + residual[r, n]
        out = 0 if relu and z < 0 else z     (NaN stays NaN)

    scale None = 1, shift None = 0, residual None = 0.  residual holds float32
    (res_dt F32) or bf16 bits (BF16), [n_out, C_out].  Returns (out, bound)
    in float64, unrounded; bound = |scale| absb + |shift| + |residual| scales
    the rounding error of the fused result (ReLU is 1-Lipschitz).
    """
    y = np.asarray(y, dtype=np.float64)
    absb = np.asarray(absb, dtype=np.float64)
    z = y.copy()
    bound = absb.copy()
    if scale is not None:
        sc = np.asarray(scale, dtype=np.float32).astype(np.float64)
        z = z * sc
        bound = bound * np.abs(sc)
    if shift is not None:
        sh = np.asarray(shift, dtype=np.float32).astype(np.float64)
        z = z + sh
        bound = bound + np.abs(sh)
    if residual is not None:
        r = np.asarray(residual)
        if res_dt == BF16:
            r = (r.astype(np.uint32) << 16).view(np.float32)
        r = r.astype(np.float64)
        z = z + r
        bound = bound + np.abs(r)
    if relu:
        z = np.where(z < 0, 0.0, z)
    return z, bound


def round_to(v, out_dt):
    """Round a float64 array once to fp32 (float32) or bf16 (uint16 bits)."""
    lib = _load()
    v = np.ascontiguousarray(v, dtype=np.float64)
    out = np.empty(v.shape, np.float32 if out_dt == F32 else np.uint16)
    st = lib.ref_round(_ptr(v), v.size, out_dt, _ptr(out))
    if st != OK:
        raise OracleError(st)
    return out


def status_of_build(kind, coords, spatial_size, f, s=None):
    """Status code the oracle returns for these build arguments."""
    try:
        Rulebook(kind, coords, spatial_size, f, s)
        return OK
    except OracleError as e:
        return e.status
