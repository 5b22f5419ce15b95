"""GPU parity at the benchmark's full sizes.

Each workload is built exactly as bench.py builds it (asynchronous rule-book
build, preallocated output, the same kernels).  The oracle checks:
* the complete rule book and output site set, bit for bit (each R_i sorted
  by output row against the oracle, and in Z-order of the output site as the
  library promises);
* the features of every output row, to the same tolerances as the small
  parity tests (the oracle's forward runs on all host cores);
* the VSC invariants (k_centre = N, k_i = k_{K-1-i}) on the GPU's own counts;
* the four-level encoder stack with every book after the first chained on
  the previous SC book's device-side output sites, as bench.py runs it,
  against the oracle's own chain of books and layer outputs.
"""
import ctypes
import sys
import time

import numpy as np
import pytest

torch = pytest.importorskip("torch")

import oracle  # noqa: E402
import paper_1706_01307_amd as spc  # noqa: E402
from paper_1706_01307_amd import _lib, inputs  # noqa: E402
from tests.rb_check import check_rulebook  # noqa: E402
from tests.test_parity_gpu import (RTOL_BF16, RTOL_F32, _bf16_tensor, _t, _to_np,  # noqa: E402
                                   check_features, make_layer)

pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _bench_style_layer(kind, coords, size, f, s, x_dev, w_dev, b_dev, in_dt, out_dt, C_in,
                       C_out, out_torch_dtype):
    """Build (asynchronously) and run one layer through the raw C ABI."""
    lib = _lib.load()
    ct = _t(coords)
    D = coords.shape[1]
    h = ctypes.c_void_p()
    sz, fa, sa = (np.asarray(v, np.int32) for v in (size, f, s))
    st = lib.spconv_build_rulebook(kind, D, ctypes.c_void_p(ct.data_ptr()), len(coords),
                                   sz.ctypes.data, fa.ctypes.data, sa.ctypes.data,
                                   _lib.BUILD_ASYNC, None, ctypes.byref(h))
    assert st == 0
    rb = spc.Rulebook(h, kind, D, ctypes.c_void_p(0))
    assert rb.status() == spc.OK
    y = torch.empty((rb.n_out, C_out), dtype=out_torch_dtype, device="cuda")
    fwd = lib.spconv_vsc_forward if kind == spc.VSC else lib.spconv_sc_forward
    st = fwd(h, in_dt, ctypes.c_void_p(x_dev.data_ptr()), ctypes.c_void_p(w_dev.data_ptr()),
             ctypes.c_void_p(b_dev.data_ptr()), out_dt, ctypes.c_void_p(y.data_ptr()), C_in,
             C_out, None)
    assert st == 0
    torch.cuda.synchronize()
    return rb, y


def _full_check(name, seed=11):
    t0 = time.time()
    wl = inputs.make_workload(name)
    layer = wl.layers[0]
    N, D = len(wl.coords), wl.d + 1
    K = layer.f ** wl.d
    _say(f"[{name}] N={N} generated in {time.time() - t0:.1f}s")
    bf16 = wl.dtype == "bf16"
    xf = inputs.normal_f32((N, layer.c_in), seed=seed)
    w, b = make_layer(seed + 1, K, layer.c_in, layer.c_out, wl.dtype)
    if bf16:
        x = inputs.to_bf16_bits(xf)
        xd, wd = _bf16_tensor(x), _bf16_tensor(w)
        in_dt = out_dt = _lib.BF16
        od = torch.bfloat16
    else:
        x = xf
        xd, wd = _t(x), _t(w)
        in_dt = out_dt = _lib.F32
        od = torch.float32
    f = [1] + [layer.f] * wl.d
    rb, y = _bench_style_layer(spc.VSC, wl.coords, wl.spatial_size, f, [1] * D, xd, wd, _t(b),
                               in_dt, out_dt, layer.c_in, layer.c_out, od)
    _say(f"[{name}] GPU done; oracle rule book ...")
    t0 = time.time()
    ref = oracle.Rulebook(oracle.VSC, wl.coords, wl.spatial_size, f)
    _say(f"[{name}] oracle rule book {time.time() - t0:.1f}s, sum k = {ref.pair_off[-1]}")
    off = rb.pair_off
    k = np.diff(off)
    assert k[K // 2] == N and np.array_equal(k, k[::-1])
    oc, pairs = rb.export()
    check_rulebook(oc.cpu().numpy(), pairs.cpu().numpy(), off, ref)
    t0 = time.time()
    yo, absb = ref.forward(x, w, b, in_dt=oracle.BF16 if bf16 else oracle.F32)
    _say(f"[{name}] oracle forward {time.time() - t0:.1f}s on {oracle.set_threads(0)} threads")
    check_features(_to_np(y), yo, absb, RTOL_BF16 if bf16 else RTOL_F32, name)
    _say(f"[{name}] rule book exact, all {N} rows within tolerance")
    return rb, y


def test_fullsize_headline_surf128x8_c64_bf16():
    rb, y = _full_check("surf128x8_vsc3_c64_bf16")
    # bitwise repeatability of the full output at this size
    y0 = y.view(torch.int16).clone()
    rb2, y2 = _full_check("surf128x8_vsc3_c64_bf16")
    assert torch.equal(y0, y2.view(torch.int16))


def test_fullsize_headline_on_the_hashed_site_map(monkeypatch):
    """The headline book built on the hashed site map (sorted bricks: the
    sites sorted by their brick bits only, two 9-bit radix passes, each
    brick's run put in cell order by the pool fill) is the oracle's, bit for
    bit, and its forward equals the dense grid's bit for bit; a duplicate
    site placed far from its twin in the input is reported."""
    wl = inputs.make_workload("surf128x8_vsc3_c64_bf16")
    N = len(wl.coords)
    f = [1, 3, 3, 3]
    x = _bf16_tensor(inputs.to_bf16_bits(inputs.normal_f32((N, 64), seed=61)))
    w, b = make_layer(62, 27, 64, 64, "bf16")
    wd, bd = _bf16_tensor(w), _t(b)
    monkeypatch.setenv("SPCONV_RULEBOOK", "grid")
    rbg = spc.build_rulebook(spc.VSC, _t(wl.coords), wl.spatial_size, f)
    yg = spc.vsc_forward(rbg, x, wd, bd)
    monkeypatch.setenv("SPCONV_RULEBOOK", "hash")
    rbh = spc.build_rulebook(spc.VSC, _t(wl.coords), wl.spatial_size, f)
    yh = spc.vsc_forward(rbh, x, wd, bd)
    torch.cuda.synchronize()
    assert torch.equal(yg.view(torch.int16), yh.view(torch.int16))
    ref = oracle.Rulebook(oracle.VSC, wl.coords, wl.spatial_size, f)
    oc, pairs = rbh.export()
    check_rulebook(oc.cpu().numpy(), pairs.cpu().numpy(), rbh.pair_off, ref)
    _say(f"[hash headline] N={N}: book exact, forward equal to the grid's")
    dup = np.concatenate([wl.coords, wl.coords[N // 3:N // 3 + 1]], axis=0)
    st = spc.build_rulebook(spc.VSC, _t(dup), wl.spatial_size, f, sync=False).status()
    assert st == spc.EDUP


def test_fullsize_surf64x16_c32_f32():
    _full_check("surf64x16_vsc3_c32")


def test_fullsize_pen64_c1x16_f32():
    wl = inputs.make_workload("pen64_vsc3_c1x16")
    x = np.ones((len(wl.coords), 1), np.float32)
    w, b = make_layer(3, 9, 1, 16, "f32")
    rb = spc.build_rulebook(spc.VSC, _t(wl.coords), wl.spatial_size, [1, 3, 3])
    y = spc.vsc_forward(rb, _t(x), _t(w), _t(b))
    ref = oracle.Rulebook(oracle.VSC, wl.coords, wl.spatial_size, [1, 3, 3])
    oc, pairs = rb.export()
    check_rulebook(oc.cpu().numpy(), pairs.cpu().numpy(), rb.pair_off, ref)
    yo, absb = ref.forward(x, w, b)
    check_features(_to_np(y), yo, absb, RTOL_F32, "pen64")


def test_fullsize_pen_stack_64_grids():
    """VSC 1->32->32->32 on one rule book, then SC 2x2/2, on 64 grids."""
    wl = inputs.make_workload("pen64x64_vsc3x3_sc2")
    size = wl.spatial_size
    ref_v = oracle.Rulebook(oracle.VSC, wl.coords, size, [1, 3, 3])
    rb = spc.build_rulebook(spc.VSC, _t(wl.coords), size, [1, 3, 3])
    oc, pairs = rb.export()
    check_rulebook(oc.cpu().numpy(), pairs.cpu().numpy(), rb.pair_off, ref_v)
    x = np.ones((len(wl.coords), 1), np.float32)
    xg, xo, xa = _t(x), x, np.abs(x).astype(np.float64)
    for li, lay in enumerate(wl.layers[:3]):
        w, b = make_layer(20 + li, 9, lay.c_in, lay.c_out, "f32")
        xg = spc.vsc_forward(rb, xg, _t(w), _t(b))
        yo, absb = ref_v.forward(xo, w, b, x_absb=xa)
        check_features(_to_np(xg), yo, absb, RTOL_F32, f"stack {li}")
        xo, xa = oracle.round_to(yo, oracle.F32), absb
    lay = wl.layers[3]
    w, b = make_layer(30, 4, lay.c_in, lay.c_out, "f32")
    rbs = spc.build_rulebook(spc.SC, _t(wl.coords), size, [1, 2, 2], [1, 2, 2])
    ys = spc.sc_forward(rbs, xg, _t(w), _t(b))
    ref_s = oracle.Rulebook(oracle.SC, wl.coords, size, [1, 2, 2], [1, 2, 2])
    oc, pairs = rbs.export()
    check_rulebook(oc.cpu().numpy(), pairs.cpu().numpy(), rbs.pair_off, ref_s)
    yo, absb = ref_s.forward(xo, w, b, x_absb=xa)
    check_features(_to_np(ys), yo, absb, RTOL_F32, "stack SC")


def test_fullsize_encoder_level0_and_downsample():
    """256^3 x 4 surfaces: level-0 VSC (32->32, bf16) and the 2^3 stride-2 SC
    to level 1 built from the generated sites: rule books exact, every row of
    both layers within tolerance."""
    t0 = time.time()
    wl = inputs.make_workload("surf256x4_unet_enc_bf16")
    N = len(wl.coords)
    _say(f"[encoder] N={N} generated in {time.time() - t0:.1f}s")
    size = wl.spatial_size
    x = inputs.to_bf16_bits(inputs.normal_f32((N, 32), seed=5))
    w, b = make_layer(40, 27, 32, 32, "bf16")
    rb, y = _bench_style_layer(spc.VSC, wl.coords, size, [1, 3, 3, 3], [1, 1, 1, 1],
                               _bf16_tensor(x), _bf16_tensor(w), _t(b), _lib.BF16, _lib.BF16,
                               32, 32, torch.bfloat16)
    ref = oracle.Rulebook(oracle.VSC, wl.coords, size, [1, 3, 3, 3])
    _say(f"[encoder] oracle VSC rule book done ({time.time() - t0:.1f}s)")
    oc, pairs = rb.export()
    check_rulebook(oc.cpu().numpy(), pairs.cpu().numpy(), rb.pair_off, ref)
    yo, absb = ref.forward(x, w, b, in_dt=oracle.BF16)
    check_features(_to_np(y), yo, absb, RTOL_BF16, "encoder L0 VSC")
    del ref, yo, absb
    # SC 2^3 stride 2 from the generated input (32 -> 64)
    w2, b2 = make_layer(41, 8, 32, 64, "bf16")
    rbs, ys = _bench_style_layer(spc.SC, wl.coords, size, [1, 2, 2, 2], [1, 2, 2, 2],
                                 _bf16_tensor(x), _bf16_tensor(w2), _t(b2), _lib.BF16, _lib.BF16,
                                 32, 64, torch.bfloat16)
    refs = oracle.Rulebook(oracle.SC, wl.coords, size, [1, 2, 2, 2], [1, 2, 2, 2])
    _say(f"[encoder] oracle SC rule book done, n_out = {refs.n_out}")
    oc, pairs = rbs.export()
    check_rulebook(oc.cpu().numpy(), pairs.cpu().numpy(), rbs.pair_off, refs)
    yo, absb = refs.forward(x, w2, b2, in_dt=oracle.BF16)
    check_features(_to_np(ys), yo, absb, RTOL_BF16, "encoder SC")
    _say(f"[encoder] level 0 done ({time.time() - t0:.1f}s)")


def test_fullsize_encoder_stack_chained():
    """The whole four-level encoder (levels at C = 32/64/96/128, two VSC 3^3
    layers per level, 2^3 stride-2 SC between levels, bf16) enqueued as
    bench.py's stack mode does: asynchronous builds, every book after the
    first level's built on the previous SC book's output sites and device-side
    count (spconv_build_rulebook_on), feature buffers sized by the books' row
    bounds.  Against the oracle's own chain: each level's VSC and SC books are
    built by the oracle on the oracle's SC output sites and must match bit
    for bit; each layer's output is compared on every row with the oracle's
    forward of the oracle's own previous output (rounded to bf16 as the GPU
    stores it), the absolute-sum bound carried through the layers."""
    t0 = time.time()
    wl = inputs.make_workload("surf256x4_unet_enc_bf16")
    lib = _lib.load()
    D = wl.d + 1
    N0 = len(wl.coords)
    ct = _t(wl.coords)
    x_bits = inputs.to_bf16_bits(inputs.normal_f32((N0, wl.layers[0].c_in), seed=11))
    xg = _bf16_tensor(x_bits)
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    # ---- GPU: enqueue everything without waiting
    books, outs, handles = [], [], []
    rb, parent = None, None
    params, dev_params = [], []
    for j, L in enumerate(wl.layers):
        K = L.f ** wl.d
        w, b = make_layer(300 + 2 * j, K, L.c_in, L.c_out, "bf16")
        params.append((w, b))
        dev_params.append((_bf16_tensor(w), _t(b)))     # alive until the chain has run
        f = np.array([1] + [L.f] * wl.d, np.int32)
        s = np.array([1] + [L.s] * wl.d, np.int32)
        kind = _lib.VSC if L.kind == "vsc" else _lib.SC
        h = rb if L.kind == "vsc" else None
        if h is None:
            h = ctypes.c_void_p()
            if parent is not None:
                st = lib.spconv_build_rulebook_on(parent, kind, f.ctypes.data, s.ctypes.data,
                                                  _lib.BUILD_ASYNC, stream, ctypes.byref(h))
            else:
                sz = np.array(wl.spatial_size, np.int32)
                st = lib.spconv_build_rulebook(kind, D, ctypes.c_void_p(ct.data_ptr()), N0,
                                               sz.ctypes.data, f.ctypes.data, s.ctypes.data,
                                               _lib.BUILD_ASYNC, stream, ctypes.byref(h))
            assert st == 0, (j, st)
            handles.append(h)
        nb_in, nb_out = ctypes.c_int64(), ctypes.c_int64()
        assert lib.spconv_rulebook_bounds(h, ctypes.byref(nb_in), ctypes.byref(nb_out)) == 0
        y = torch.empty((nb_out.value, L.c_out), dtype=torch.bfloat16, device="cuda")
        fwd = lib.spconv_vsc_forward if L.kind == "vsc" else lib.spconv_sc_forward
        wd, bd = dev_params[-1]
        st = fwd(h, _lib.BF16, ctypes.c_void_p(xg.data_ptr()), ctypes.c_void_p(wd.data_ptr()),
                 ctypes.c_void_p(bd.data_ptr()), _lib.BF16, ctypes.c_void_p(y.data_ptr()),
                 L.c_in, L.c_out, stream)
        assert st == 0, (j, st)
        books.append(h)
        outs.append(y)
        if L.kind == "vsc":
            rb = h
        else:
            rb, parent = None, h
        xg = y
    torch.cuda.synchronize()
    _say(f"[stack] GPU chain enqueued and done ({time.time() - t0:.1f}s)")
    # ---- oracle chain, layer by layer
    coords, size = wl.coords, np.array(wl.spatial_size)
    xo, xa = x_bits, None
    ref_v = None
    for j, L in enumerate(wl.layers):
        w, b = params[j]
        h = books[j]
        if L.kind == "vsc":
            if ref_v is None:
                ref_v = oracle.Rulebook(oracle.VSC, coords, size, [1] + [L.f] * wl.d)
            ref = ref_v
        else:
            ref = oracle.Rulebook(oracle.SC, coords, size, [1] + [L.f] * wl.d,
                                  [1] + [L.s] * wl.d)
        g = spc.Rulebook(h, spc.SC if L.kind == "sc" else spc.VSC, D, stream)
        assert g.status() == spc.OK
        assert g.n_in == ref.n_in and g.n_out == ref.n_out, (j, g.n_in, g.n_out)
        if L.kind == "sc" or j == 0 or wl.layers[j - 1].kind == "sc":
            oc, pairs = g.export()
            check_rulebook(oc.cpu().numpy(), pairs.cpu().numpy(), g.pair_off, ref)
        g._h = None                      # the handles are destroyed below
        yo, absb = ref.forward(xo, w, b, in_dt=oracle.BF16, x_absb=xa)
        check_features(_to_np(outs[j][:ref.n_out]), yo, absb, RTOL_BF16, f"stack layer {j}")
        _say(f"[stack] layer {j} ({L.kind} {L.c_in}->{L.c_out}, {ref.n_out} rows, "
             f"sum k {ref.pair_off[-1]}) matches ({time.time() - t0:.1f}s)")
        xo, xa = oracle.round_to(yo, oracle.BF16), absb
        if L.kind == "sc":
            coords, size, ref_v = ref.out_coords, ref.out_size, None
    for h in handles:
        lib.spconv_rulebook_destroy(h)
