"""GPU parity of sparse pooling, DC and the gradients against the oracle.

* MP is exact (a maximum of the zero vector and input values), so it is
  compared bit for bit; AP and everything with products use the features
  bound of the forward tests: per element |g - o| <= rtol * S and normwise
  ||g - o|| <= rtol ||o||, with rtol 1e-5 (fp32) / 2e-2 (bf16 in or out).
* Weight and bias gradients sum up to k_i products per entry in fp32, in
  chunks of at most 4096 pairs whose partial sums are then added in order; their
  tolerance is RTOL_GRAD = 1e-4, ~25x the typical sqrt(n) * 2^-24 error of a
  4096-term fp32 sum (the worst case n * 2^-24 is 2.4e-4).
"""
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")

import oracle  # noqa: E402
import paper_1706_01307_amd as spc  # noqa: E402
from paper_1706_01307_amd import inputs  # noqa: E402
from tests.test_parity_gpu import (RTOL_BF16, RTOL_F32, _bf16_tensor, _t,  # noqa: E402
                                   _to_np, check_features)

pytestmark = pytest.mark.gpu

RTOL_GRAD = 1e-4
OP = {"vsc": (spc.OP_VSC, oracle.VSC), "sc": (spc.OP_SC, oracle.SC), "dc": (spc.OP_DC, oracle.DC)}


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.init()


def _feats(n, C, dtype, seed, std=1.0):
    f = inputs.normal_f32((n, C), std=std, seed=seed)
    return inputs.to_bf16_bits(f) if dtype == "bf16" else f


def _dev(a, dtype):
    return _bf16_tensor(a) if dtype == "bf16" else _t(a)


def _odt(dtype):
    return oracle.BF16 if dtype == "bf16" else oracle.F32


def _pen(n_grids, seed):
    return inputs.pen_strokes(n_grids, 64, seed=seed), [n_grids, 64, 64]


def _surf(n, size, seed):
    c = inputs.surfaces(n, size, size / 8, size * 0.45, seed=seed, variant="literal")
    return c, [n, size, size, size]


def _sites(case):
    if case == "pen":
        return _pen(16, 3)
    if case == "surf":
        return _surf(2, 48, 5)
    raise ValueError(case)


# ---------------------------------------------------------------------------
# Pooling
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("case,f,s,C,dtype", [
    ("pen", [1, 2, 2], [1, 2, 2], 32, "f32"),
    ("pen", [1, 3, 3], [1, 2, 2], 5, "f32"),
    ("pen", [1, 2, 3], [1, 2, 3], 16, "bf16"),
    ("surf", [1, 2, 2, 2], [1, 2, 2, 2], 32, "bf16"),
    ("surf", [1, 3, 3, 3], [1, 2, 2, 2], 8, "f32"),
])
def test_pool_matches_oracle(case, f, s, C, dtype):
    coords, size = _sites(case)
    _say(f"[pool] {case} N={len(coords)} f={f} s={s} C={C} {dtype}")
    x = _feats(len(coords), C, dtype, 41)
    rb = spc.build_rulebook(spc.SC, _t(coords), size, f, s)
    ref = oracle.Rulebook(oracle.SC, coords, size, f, s)
    xd = _dev(x, dtype)
    mp = spc.pool_forward(rb, xd, spc.POOL_MAX)
    ap = spc.pool_forward(rb, xd, spc.POOL_AVG)
    torch.cuda.synchronize()
    mo, _ = ref.pool(x, oracle.POOL_MAX, _odt(dtype))
    ao, absb = ref.pool(x, oracle.POOL_AVG, _odt(dtype))
    want = oracle.round_to(mo, _odt(dtype))
    got = mp.view(torch.int16).cpu().numpy().view(np.uint16) if dtype == "bf16" else mp.cpu().numpy()
    np.testing.assert_array_equal(got, want)
    check_features(_to_np(ap), ao, absb, RTOL_F32 if dtype == "f32" else RTOL_BF16, "AP")


def test_pool_max_ignores_nan_and_empty_input():
    coords, size = _pen(2, 9)
    x = _feats(len(coords), 8, "f32", 3)
    x[5, 2] = np.nan
    x[17, :] = np.nan
    rb = spc.build_rulebook(spc.SC, _t(coords), size, [1, 2, 2], [1, 2, 2])
    got = spc.pool_forward(rb, _t(x), spc.POOL_MAX).cpu().numpy()
    ref = oracle.Rulebook(oracle.SC, coords, size, [1, 2, 2], [1, 2, 2])
    want = ref.pool(x, oracle.POOL_MAX)[0].astype(np.float32)
    assert not np.isnan(got).any()
    np.testing.assert_array_equal(got, want)
    empty = spc.build_rulebook(spc.SC, _t(np.zeros((0, 3), np.int32)), size, [1, 2, 2], [1, 2, 2])
    out = spc.pool_forward(empty, torch.zeros((0, 8), device="cuda"), spc.POOL_AVG)
    assert out.shape == (0, 8)


# ---------------------------------------------------------------------------
# Deconvolution
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("case,f,s,C_in,C_out,dtype", [
    ("pen", [1, 2, 2], [1, 2, 2], 32, 32, "f32"),
    ("pen", [1, 3, 3], [1, 2, 2], 1, 16, "f32"),
    ("pen", [1, 3, 3], [1, 2, 2], 16, 16, "f32"),
    ("surf", [1, 2, 2, 2], [1, 2, 2, 2], 32, 32, "bf16"),
    ("surf", [1, 2, 2, 2], [1, 2, 2, 2], 64, 32, "bf16"),
    ("surf", [1, 3, 3, 3], [1, 2, 2, 2], 32, 16, "f32"),
])
def test_dc_matches_oracle(case, f, s, C_in, C_out, dtype):
    coords, size = _sites(case)
    K = int(np.prod(f))
    rb = spc.build_rulebook(spc.SC, _t(coords), size, f, s, transpose=True)
    ref = oracle.Rulebook(oracle.SC, coords, size, f, s)
    _say(f"[dc] {case} N={len(coords)} -> {ref.n_out} f={f} s={s} C={C_in}->{C_out} {dtype}")
    x = _feats(ref.n_out, C_in, dtype, 51)
    wf = inputs.normal_f32((K, C_in, C_out), std=1.0 / np.sqrt(K * C_in), seed=52)
    w = inputs.to_bf16_bits(wf) if dtype == "bf16" else wf
    b = inputs.normal_f32((C_out,), std=0.1, seed=53)
    y = spc.dc_forward(rb, _dev(x, dtype), _dev(w, dtype), _t(b))
    yo, absb = ref.dc_forward(x, w, b, in_dt=_odt(dtype))
    check_features(_to_np(y), yo, absb, RTOL_F32 if dtype == "f32" else RTOL_BF16, "DC")
    y2 = spc.dc_forward(rb, _dev(x, dtype), _dev(w, dtype), _t(b))
    assert torch.equal(y, y2)                    # bitwise reproducible


def test_dc_needs_the_transposed_book():
    coords, size = _pen(2, 4)
    rb = spc.build_rulebook(spc.SC, _t(coords), size, [1, 2, 2], [1, 2, 2])
    x = torch.zeros((rb.n_out, 16), device="cuda")
    w = torch.zeros((4, 16, 16), device="cuda")
    with pytest.raises(spc.SpconvError):
        spc.dc_forward(rb, x, w)
    with pytest.raises(spc.SpconvError):
        spc.backward_data(rb, spc.OP_SC, torch.zeros((rb.n_out, 16), device="cuda"), w)


# ---------------------------------------------------------------------------
# Gradients
# ---------------------------------------------------------------------------

GRAD_CASES = [
    ("vsc", "pen", [1, 3, 3], None, 32, 32, "f32"),
    ("vsc", "pen", [1, 3, 3], None, 1, 16, "f32"),
    ("vsc", "surf", [1, 3, 3, 3], None, 32, 32, "bf16"),
    ("vsc", "surf", [1, 3, 3, 3], None, 64, 64, "bf16"),
    ("vsc", "surf", [1, 3, 3, 3], None, 16, 32, "f32"),
    ("sc", "pen", [1, 2, 2], [1, 2, 2], 32, 32, "f32"),
    ("sc", "pen", [1, 3, 3], [1, 2, 2], 16, 32, "bf16"),
    ("sc", "surf", [1, 2, 2, 2], [1, 2, 2, 2], 32, 64, "bf16"),
    ("dc", "pen", [1, 2, 2], [1, 2, 2], 32, 16, "f32"),
    ("dc", "surf", [1, 2, 2, 2], [1, 2, 2, 2], 64, 32, "bf16"),
    ("vsc", "surf", [1, 3, 3, 3], None, 32, 96, "bf16"),
    ("sc", "pen", [1, 2, 2], [1, 2, 2], 3, 5, "f32"),
    # input gradients with at most 4 gradient planes on 16-column outputs
    # (the few-input-plane kernel, transposed weights)
    ("vsc", "pen", [1, 3, 3], None, 16, 2, "f32"),
    ("sc", "pen", [1, 2, 2], [1, 2, 2], 32, 4, "bf16"),
    ("dc", "pen", [1, 2, 2], [1, 2, 2], 3, 16, "f32"),
]


def _grad_setup(op, case, f, s, C_in, C_out, dtype):
    coords, size = _sites(case)
    kind = spc.VSC if op == "vsc" else spc.SC
    s = s or [1] * len(f)
    rb = spc.build_rulebook(kind, _t(coords), size, f, s, transpose=(op == "sc"))
    ref = oracle.Rulebook(kind, coords, size, f, s)
    in_rows = ref.n_out if op == "dc" else ref.n_in
    out_rows = ref.n_in if op == "dc" else ref.n_out
    K = ref.K
    x = _feats(in_rows, C_in, dtype, 61)
    dy = _feats(out_rows, C_out, dtype, 62)
    wf = inputs.normal_f32((K, C_in, C_out), std=1.0 / np.sqrt(K * C_in), seed=63)
    w = inputs.to_bf16_bits(wf) if dtype == "bf16" else wf
    return coords, rb, ref, x, dy, w


@pytest.mark.parametrize("op,case,f,s,C_in,C_out,dtype", GRAD_CASES)
def test_input_gradient_matches_oracle(op, case, f, s, C_in, C_out, dtype):
    coords, rb, ref, x, dy, w = _grad_setup(op, case, f, s, C_in, C_out, dtype)
    _say(f"[dx] {op} {case} N={len(coords)} f={f} C={C_in}->{C_out} {dtype}")
    dx = spc.backward_data(rb, OP[op][0], _dev(dy, dtype), _dev(w, dtype))
    dxo, absb = ref.backward_data(OP[op][1], dy, w, _odt(dtype))
    check_features(_to_np(dx), dxo, absb, RTOL_F32 if dtype == "f32" else RTOL_BF16, "dx")
    dx2 = spc.backward_data(rb, OP[op][0], _dev(dy, dtype), _dev(w, dtype))
    assert torch.equal(dx, dx2)


@pytest.mark.parametrize("op,case,f,s,C_in,C_out,dtype", GRAD_CASES)
def test_weight_gradient_matches_oracle(op, case, f, s, C_in, C_out, dtype):
    coords, rb, ref, x, dy, w = _grad_setup(op, case, f, s, C_in, C_out, dtype)
    _say(f"[dw] {op} {case} N={len(coords)} f={f} C={C_in}->{C_out} {dtype}")
    dw, db = spc.backward_weight(rb, OP[op][0], _dev(x, dtype), _dev(dy, dtype), C_in, C_out)
    dwo, dbo, aw, ab = ref.backward_weight(OP[op][1], x, dy, C_in, C_out, _odt(dtype))
    check_features(dw.cpu().numpy(), dwo, aw, RTOL_GRAD, "dw")
    check_features(db.cpu().numpy(), dbo, ab, RTOL_GRAD, "db")
    dw2, db2 = spc.backward_weight(rb, OP[op][0], _dev(x, dtype), _dev(dy, dtype), C_in, C_out)
    assert torch.equal(dw, dw2) and torch.equal(db, db2)


def test_gradient_op_must_match_the_book():
    coords, size = _pen(2, 6)
    vsc = spc.build_rulebook(spc.VSC, _t(coords), size, [1, 3, 3])
    w = torch.zeros((9, 8, 8), device="cuda")
    dy = torch.zeros((len(coords), 8), device="cuda")
    for op in (spc.OP_SC, spc.OP_DC):
        with pytest.raises(spc.SpconvError):
            spc.backward_data(vsc, op, dy, w)
        with pytest.raises(spc.SpconvError):
            spc.backward_weight(vsc, op, dy, dy, 8, 8)


# ---------------------------------------------------------------------------
# Forward with the block epilogue fused (affine per channel, residual, ReLU)
# ---------------------------------------------------------------------------

FUSED_CASES = [
    # kind, case, f, s, C_in, C_out, dtype, out dtype
    ("vsc", "surf", [1, 3, 3, 3], [1, 1, 1, 1], 64, 64, "bf16", "bf16"),
    ("vsc", "surf", [1, 3, 3, 3], [1, 1, 1, 1], 32, 32, "f32", "f32"),
    ("vsc", "pen", [1, 3, 3], [1, 1, 1], 1, 16, "f32", "f32"),        # few input planes
    ("vsc", "pen", [1, 3, 3], [1, 1, 1], 3, 32, "bf16", "f32"),       # few input planes
    ("vsc", "pen", [1, 3, 3], [1, 1, 1], 16, 24, "bf16", "f32"),      # vector path
    ("vsc", "pen", [1, 3, 3], [1, 1, 1], 32, 32, "bf16", "bf16"),     # 2 column blocks
    ("sc", "surf", [1, 2, 2, 2], [1, 2, 2, 2], 32, 64, "bf16", "bf16"),
    ("sc", "pen", [1, 3, 3], [1, 2, 2], 32, 16, "f32", "bf16"),       # 1 column block
]
PARTS = {"all": (1, 1, 1, 1), "affine": (1, 1, 0, 0), "res_relu": (0, 0, 1, 1),
         "scale_relu": (1, 0, 0, 1)}


def _fused_setup(kind, case, f, s, C_in, C_out, dtype, out_dtype):
    coords, size = _sites(case)
    K = int(np.prod(f))
    sk, ok = (spc.VSC, oracle.VSC) if kind == "vsc" else (spc.SC, oracle.SC)
    rb = spc.build_rulebook(sk, _t(coords), size, f, s)
    ref = oracle.Rulebook(ok, coords, size, f, s)
    x = _feats(len(coords), C_in, dtype, 61)
    wf = inputs.normal_f32((K, C_in, C_out), std=1.0 / np.sqrt(K * C_in), seed=62)
    w = inputs.to_bf16_bits(wf) if dtype == "bf16" else wf
    scale = inputs.normal_f32((C_out,), std=1.0, seed=63)
    shift = inputs.normal_f32((C_out,), std=0.5, seed=64)
    res = _feats(ref.n_out, C_out, out_dtype, 65)
    return coords, rb, ref, x, w, scale, shift, res


@pytest.mark.parametrize("parts", list(PARTS))
@pytest.mark.parametrize("kind,case,f,s,C_in,C_out,dtype,out_dtype", FUSED_CASES)
def test_fused_forward_matches_oracle(kind, case, f, s, C_in, C_out, dtype, out_dtype, parts):
    coords, rb, ref, x, w, scale, shift, res = _fused_setup(kind, case, f, s, C_in, C_out, dtype,
                                                            out_dtype)
    use_s, use_b, use_r, relu = PARTS[parts]
    _say(f"[fused] {kind} {case} N={len(coords)} f={f} s={s} C={C_in}->{C_out} {dtype}->"
         f"{out_dtype} {parts}")
    odt = torch.bfloat16 if out_dtype == "bf16" else torch.float32
    y = spc.forward_fused(rb, _dev(x, dtype), _dev(w, dtype),
                          scale=_t(scale) if use_s else None, shift=_t(shift) if use_b else None,
                          residual=_dev(res, out_dtype) if use_r else None, relu=bool(relu),
                          out_dtype=odt)
    y64, absb = ref.forward(x, w, None, in_dt=_odt(dtype))
    zo, bound = oracle.fused_epilogue(y64, absb, scale if use_s else None,
                                      shift if use_b else None, res if use_r else None,
                                      bool(relu), _odt(out_dtype))
    rtol = RTOL_F32 if dtype == "f32" and out_dtype == "f32" else RTOL_BF16
    g = _to_np(y)
    check_features(g, zo, bound, rtol, "fused")
    if relu:
        assert (g >= 0).all()


def test_fused_forward_reduces_to_the_plain_forward():
    """scale = residual = NULL, no ReLU: bit for bit the forward with bias."""
    for args in (FUSED_CASES[0], FUSED_CASES[2], FUSED_CASES[5]):
        kind, case, f, s, C_in, C_out, dtype, out_dtype = args
        _, rb, _, x, w, _, shift, _ = _fused_setup(*args)
        odt = torch.bfloat16 if out_dtype == "bf16" else torch.float32
        fwd = spc.vsc_forward if kind == "vsc" else spc.sc_forward
        y0 = fwd(rb, _dev(x, dtype), _dev(w, dtype), _t(shift), out_dtype=odt)
        y1 = spc.forward_fused(rb, _dev(x, dtype), _dev(w, dtype), shift=_t(shift), out_dtype=odt)
        assert torch.equal(y0, y1), args


def test_fused_forward_in_place_residual_and_overlap_errors():
    args = FUSED_CASES[0]
    kind, case, f, s, C_in, C_out, dtype, out_dtype = args
    _, rb, ref, x, w, scale, shift, res = _fused_setup(*args)
    xd, wd = _dev(x, dtype), _dev(w, dtype)
    r = _dev(res, out_dtype)
    y = spc.forward_fused(rb, xd, wd, _t(scale), _t(shift), r, True)
    buf = r.clone()
    y2 = spc.forward_fused(rb, xd, wd, _t(scale), _t(shift), buf, True, out=buf)
    assert y2.data_ptr() == buf.data_ptr()
    assert torch.equal(y, y2)
    n = ref.n_out * C_out
    big = torch.zeros(2 * n + 64, dtype=torch.bfloat16, device="cuda")
    out = big[:n].view(ref.n_out, C_out)
    shifted = big[64:64 + n].view(ref.n_out, C_out)     # overlaps out, not equal to it
    with pytest.raises(spc.SpconvError):
        spc.forward_fused(rb, xd, wd, residual=shifted, out=out)
    lib = spc._lib.load()
    ptr = out.data_ptr()
    st = lib.spconv_forward_fused(rb.handle, spc.BF16, xd.data_ptr(), wd.data_ptr(), None, None,
                                  ptr + 2 * n + 8, 0, spc.BF16, ptr, C_in, C_out, None)
    assert st == spc._lib.EINVAL                       # residual not 16-byte aligned
    st = lib.spconv_forward_fused(rb.handle, spc.BF16, xd.data_ptr(), wd.data_ptr(), None, None,
                                  None, 2, spc.BF16, ptr, C_in, C_out, None)
    assert st == spc._lib.EINVAL                       # relu not 0 / 1


def test_empty_and_single_site_books():
    """No sites: every op returns empty (or zero) results without launching
    anything out of range.  One site: only the centre offset has a pair, so
    the weight gradient is x^T dy at the centre and zero elsewhere."""
    size = [1, 16, 16]
    none = np.zeros((0, 3), np.int32)
    vsc = spc.build_rulebook(spc.VSC, _t(none), size, [1, 3, 3])
    sc = spc.build_rulebook(spc.SC, _t(none), size, [1, 2, 2], [1, 2, 2], transpose=True)
    w = torch.zeros((9, 16, 32), device="cuda")
    x0 = torch.zeros((0, 16), device="cuda")
    assert spc.forward_fused(vsc, x0, w, relu=True).shape == (0, 32)
    assert spc.backward_data(vsc, spc.OP_VSC, torch.zeros((0, 32), device="cuda"), w).shape == (0, 16)
    dw, db = spc.backward_weight(vsc, spc.OP_VSC, x0, torch.zeros((0, 32), device="cuda"), 16, 32)
    assert dw.shape == (9, 16, 32) and not dw.any() and not db.any()
    assert spc.dc_forward(sc, x0, torch.zeros((4, 16, 32), device="cuda")).shape == (0, 32)

    one = np.array([[0, 7, 9]], np.int32)
    rb = spc.build_rulebook(spc.VSC, _t(one), size, [1, 3, 3])
    x = inputs.normal_f32((1, 16), seed=71)
    dy = inputs.normal_f32((1, 32), seed=72)
    dw, db = spc.backward_weight(rb, spc.OP_VSC, _t(x), _t(dy), 16, 32)
    dw = dw.cpu().numpy()
    np.testing.assert_allclose(dw[4], np.outer(x[0], dy[0]), rtol=1e-6, atol=0)
    assert not np.delete(dw, 4, axis=0).any()
    np.testing.assert_array_equal(db.cpu().numpy(), dy[0])


# ---------------------------------------------------------------------------
# Allocator hook
# ---------------------------------------------------------------------------

class _CountingTorchAllocator:
    """torch's caching allocator behind spconv_set_allocator, counting calls;
    fail_at = k makes the k-th allocation return NULL."""

    def __init__(self, fail_at=None):
        self.fail_at, self.calls, self.live = fail_at, 0, {}

    def alloc(self, nbytes, stream):
        self.calls += 1
        if self.fail_at == self.calls:
            return 0
        p = torch.cuda.caching_allocator_alloc(nbytes, torch.cuda.current_device(), stream)
        self.live[p] = nbytes
        return p

    def release(self, ptr, stream):
        assert ptr in self.live, "release of a pointer alloc never returned"
        del self.live[ptr]
        torch.cuda.caching_allocator_delete(ptr)


def test_allocator_hook_results_and_balance():
    coords, size = _sites("surf")
    x = _feats(len(coords), 32, "bf16", 81)
    w = inputs.to_bf16_bits(inputs.normal_f32((8, 32, 64), std=0.1, seed=82))
    ref_sc = spc.build_rulebook(spc.SC, _t(coords), size, [1, 2, 2, 2], [1, 2, 2, 2],
                                transpose=True)
    y_ref = spc.sc_forward(ref_sc, _dev(x, "bf16"), _dev(w, "bf16"))
    dx_ref = spc.backward_data(ref_sc, spc.OP_SC, y_ref, _dev(w, "bf16"))
    ref_sc.close()
    al = _CountingTorchAllocator()
    spc.set_allocator(al.alloc, al.release)
    try:
        rb = spc.build_rulebook(spc.SC, _t(coords), size, [1, 2, 2, 2], [1, 2, 2, 2],
                                transpose=True)
        assert al.calls == 3 and len(al.live) == 1     # rule book; grids and sort buffers freed
        y = spc.sc_forward(rb, _dev(x, "bf16"), _dev(w, "bf16"))
        dx = spc.backward_data(rb, spc.OP_SC, y, _dev(w, "bf16"))
        assert torch.equal(y, y_ref) and torch.equal(dx, dx_ref)
        rb.close()
        torch.cuda.synchronize()
        assert not al.live
    finally:
        spc.set_allocator(None, None)


@pytest.mark.parametrize("fail_at", [1, 2, 3])
def test_allocator_failure_is_enomem_without_leaks(fail_at):
    coords, size = _sites("pen")
    al = _CountingTorchAllocator(fail_at)
    spc.set_allocator(al.alloc, al.release)
    try:
        with pytest.raises(spc.SpconvError) as e:
            spc.build_rulebook(spc.SC, _t(coords), size, [1, 2, 2], [1, 2, 2], transpose=True)
        assert e.value.status == spc.ENOMEM
        torch.cuda.synchronize()
        assert not al.live
    finally:
        spc.set_allocator(None, None)
    rb = spc.build_rulebook(spc.SC, _t(coords), size, [1, 2, 2], [1, 2, 2], transpose=True)
    assert rb.n_out > 0                                   # the default is back


@pytest.mark.parametrize("sites,size,f,s", [
    ([[0, 4]], [1, 5], [1, 2], [1, 2]),              # f = s, the site past the last window
    ([[0, 1], [0, 2], [0, 4]], [1, 7], [1, 1], [1, 3]),  # no site on a stride multiple
])
def test_sc_book_without_outputs(sites, size, f, s):
    """An SC book whose inputs feed no output: every op accepts the empty
    tensors (NULL pointers below the ABI) and matches the oracle."""
    coords = np.asarray(sites, np.int32)
    rb = spc.build_rulebook(spc.SC, _t(coords), size, f, s, transpose=True)
    ref = oracle.Rulebook(oracle.SC, coords, size, f, s)
    assert rb.n_out == 0 == ref.n_out and rb.n_in == len(coords)
    K, ci, co = ref.K, 8, 16
    x_in = _feats(len(coords), ci, "f32", 1)
    w = inputs.normal_f32((K, ci, co), std=0.5, seed=2)
    b = inputs.normal_f32((co,), std=0.1, seed=3)
    empty_ci = torch.zeros((0, ci), device="cuda")
    empty_co = torch.zeros((0, co), device="cuda")
    assert spc.sc_forward(rb, _t(x_in), _t(w), _t(b)).shape == (0, co)
    assert spc.pool_forward(rb, _t(x_in), spc.POOL_MAX).shape == (0, ci)
    # DC from no coarse rows: the bias at every fine site
    y = spc.dc_forward(rb, empty_ci, _t(w), _t(b))
    yo, _ = ref.dc_forward(np.zeros((0, ci), np.float32), w, b, in_dt=oracle.F32)
    assert y.shape == (len(coords), co)
    np.testing.assert_array_equal(y.cpu().numpy(), yo.astype(np.float32))
    # SC input gradient from no output rows: zeros
    dx = spc.backward_data(rb, spc.OP_SC, empty_co, _t(w))
    assert dx.shape == (len(coords), ci) and not dx.abs().sum().item()
    # SC weight and bias gradients: zeros
    dw, db = spc.backward_weight(rb, spc.OP_SC, _t(x_in), empty_co, ci, co)
    assert not dw.abs().sum().item() and not db.abs().sum().item()
    # DC gradients: dy at the fine sites, no coarse rows
    dy = _feats(len(coords), co, "f32", 4)
    dw, db = spc.backward_weight(rb, spc.OP_DC, empty_ci, _t(dy), ci, co)
    dwo, dbo, aw, ab = ref.backward_weight(oracle.DC, np.zeros((0, ci), np.float32), dy, ci, co,
                                           oracle.F32)
    check_features(dw.cpu().numpy(), dwo, aw, RTOL_GRAD, "dw")
    check_features(db.cpu().numpy(), dbo, ab, RTOL_GRAD, "db")
