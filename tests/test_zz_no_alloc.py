"""spconv_backward_weight_noalloc (partials in the library's fixed scratch
array) against spconv_backward_weight with a caller workspace: the same
kernels, so the weight and bias gradients must agree bit for bit, on two
calls in a row (the second on a smaller layer, so the array holds the first
call's larger contents), and within the gradient tolerance of the oracle.
Also: a request larger than the array is rejected with ESCRATCH before any
work, and a call on a book of another device is not possible here (one GPU).
"""
import ctypes
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")

import oracle  # noqa: E402
import paper_1706_01307_amd as spc  # noqa: E402
from paper_1706_01307_amd import _lib, inputs  # noqa: E402
from tests.test_parity_gpu import _bf16_tensor, _t, check_features  # noqa: E402

pytestmark = pytest.mark.gpu
RTOL_GRAD = 1e-4


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _grads_both_ways(rb, op, x, dy, C_in, C_out, dt):
    """(dw, db) from the workspace entry and from the no-alloc entry."""
    lib = _lib.load()
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    nbytes = ctypes.c_size_t()
    _lib.check(lib.spconv_backward_weight_workspace(rb.handle, op, C_in, C_out,
                                                    ctypes.byref(nbytes)), "workspace")
    ws = torch.empty(max(nbytes.value, 16), dtype=torch.uint8, device="cuda")
    K = rb.K
    out = []
    for noalloc in (False, True):
        dw = torch.full((K, C_in, C_out), float("nan"), dtype=torch.float32, device="cuda")
        db = torch.full((C_out,), float("nan"), dtype=torch.float32, device="cuda")
        args = (rb.handle, op, dt, ctypes.c_void_p(x.data_ptr()), ctypes.c_void_p(dy.data_ptr()),
                ctypes.c_void_p(dw.data_ptr()), ctypes.c_void_p(db.data_ptr()), C_in, C_out)
        if noalloc:
            st = lib.spconv_backward_weight_noalloc(*args, stream)
        else:
            st = lib.spconv_backward_weight(*args, ctypes.c_void_p(ws.data_ptr()), nbytes.value,
                                            stream)
        _lib.check(st, "noalloc" if noalloc else "workspace")
        torch.cuda.synchronize()
        out.append((dw.cpu().numpy(), db.cpu().numpy()))
    return out


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_noalloc_matches_workspace_entry_twice(dtype):
    cases = [(inputs.surfaces(2, 64, 8, 28, seed=41, target=30000), [2, 64, 64, 64], 32, 64),
             (inputs.surfaces(1, 32, 4, 14, seed=42, target=2000), [1, 32, 32, 32], 32, 32)]
    for n, (c, size, ci, co) in enumerate(cases):
        rb = spc.build_rulebook(spc.VSC, _t(c), size, [1, 3, 3, 3])
        N = len(c)
        xf = inputs.normal_f32((N, ci), seed=50 + n)
        gf = inputs.normal_f32((N, co), seed=60 + n)
        if dtype == "bf16":
            xh, gh = inputs.to_bf16_bits(xf), inputs.to_bf16_bits(gf)
            x, g, dt, odt = _bf16_tensor(xh), _bf16_tensor(gh), _lib.BF16, oracle.BF16
        else:
            xh, gh = xf, gf
            x, g, dt, odt = _t(xf), _t(gf), _lib.F32, oracle.F32
        _say(f"[noalloc {dtype}] call {n}: N={N} C={ci}->{co}")
        (dw_ws, db_ws), (dw_na, db_na) = _grads_both_ways(rb, spc.OP_VSC, x, g, ci, co, dt)
        np.testing.assert_array_equal(dw_na, dw_ws)
        np.testing.assert_array_equal(db_na, db_ws)
        ref = oracle.Rulebook(oracle.VSC, c, size, [1, 3, 3, 3])
        dwo, dbo, aw, ab = ref.backward_weight(oracle.VSC, xh, gh, ci, co, odt)
        check_features(dw_na, dwo, aw, RTOL_GRAD, "noalloc dw")
        check_features(db_na, dbo, ab, RTOL_GRAD, "noalloc db")
        rb.close()


def test_noalloc_sc_and_dc_ops():
    """SC and DC gradients through the no-alloc entry, against the workspace
    entry (bit for bit)."""
    c = inputs.surfaces(1, 48, 6, 18, seed=43, target=5000)
    size = [1, 48, 48, 48]
    f2 = [1, 2, 2, 2]
    rb = spc.build_rulebook(spc.SC, _t(c), size, f2, f2)
    n_in, n_out = rb.n_in, rb.n_out
    a = _bf16_tensor(inputs.to_bf16_bits(inputs.normal_f32((n_in, 32), seed=1)))
    b = _bf16_tensor(inputs.to_bf16_bits(inputs.normal_f32((n_out, 32), seed=2)))
    (w1, b1), (w2, b2) = _grads_both_ways(rb, spc.OP_SC, a, b, 32, 32, _lib.BF16)
    np.testing.assert_array_equal(w1, w2)
    np.testing.assert_array_equal(b1, b2)
    (w1, b1), (w2, b2) = _grads_both_ways(rb, spc.OP_DC, b, a, 32, 32, _lib.BF16)
    np.testing.assert_array_equal(w1, w2)
    np.testing.assert_array_equal(b1, b2)


def test_noalloc_rejects_requests_beyond_the_scratch_array():
    c = inputs.surfaces(1, 64, 8, 28, seed=44, target=40000)
    rb = spc.build_rulebook(spc.VSC, _t(c), [1, 64, 64, 64], [1, 3, 3, 3])
    lib = _lib.load()
    C = 512                       # 27 offsets x 512 x 512 fp32 partials per chunk
    nbytes = ctypes.c_size_t()
    _lib.check(lib.spconv_backward_weight_workspace(rb.handle, spc.OP_VSC, C, C,
                                                    ctypes.byref(nbytes)), "workspace")
    assert nbytes.value > (128 << 20), nbytes.value
    dummy = torch.zeros(16, dtype=torch.float32, device="cuda")
    p = ctypes.c_void_p(dummy.data_ptr())
    st = lib.spconv_backward_weight_noalloc(rb.handle, spc.OP_VSC, _lib.F32, p, p, p, p, C, C,
                                            None)
    assert st == _lib.ESCRATCH
    assert "scratch" in lib.spconv_status_string(st).decode()
