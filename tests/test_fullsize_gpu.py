"""GPU parity at the benchmark's full sizes.

Each workload is built exactly as bench.py builds it (asynchronous rule-book
build, preallocated output, the same kernels).  The oracle checks:
* the complete rule book and output site set, bit for bit;
* features of a seeded sample of output rows (the oracle computes just those
  rows), to the same tolerances as the small parity tests;
* the VSC invariants (k_centre = N, k_i = k_{K-1-i}) on the GPU's own counts.
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
from tests.test_parity_gpu import (RTOL_BF16, RTOL_F32, _bf16_tensor, _t, _to_np,  # noqa: E402
                                   check_features, make_layer)

pytestmark = pytest.mark.gpu
N_SAMPLE_ROWS = 3000


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
    np.testing.assert_array_equal(off, ref.pair_off)
    _, pairs = rb.export()
    np.testing.assert_array_equal(pairs.cpu().numpy(), ref.pairs)
    rows = np.sort(np.random.default_rng(seed).choice(N, min(N, N_SAMPLE_ROWS), replace=False))
    yo, absb = ref.forward_rows(rows, x, w, b, in_dt=oracle.BF16 if bf16 else oracle.F32)
    g = _to_np(y)[rows]
    check_features(g, yo, absb, RTOL_BF16 if bf16 else RTOL_F32, name)
    _say(f"[{name}] rule book exact, {len(rows)} sampled rows within tolerance")
    return rb, y


def test_fullsize_headline_surf128x8_c64_bf16():
    rb, y = _full_check("surf128x8_vsc3_c64_bf16")
    # bitwise repeatability of the full output at this size
    y0 = y.view(torch.int16).clone()
    rb2, y2 = _full_check("surf128x8_vsc3_c64_bf16")
    assert torch.equal(y0, y2.view(torch.int16))


def test_fullsize_surf64x16_c32_f32():
    _full_check("surf64x16_vsc3_c32")


def test_fullsize_pen64_c1x16_f32():
    wl = inputs.make_workload("pen64_vsc3_c1x16")
    x = np.ones((len(wl.coords), 1), np.float32)
    w, b = make_layer(3, 9, 1, 16, "f32")
    rb = spc.build_rulebook(spc.VSC, _t(wl.coords), wl.spatial_size, [1, 3, 3])
    y = spc.vsc_forward(rb, _t(x), _t(w), _t(b))
    ref = oracle.Rulebook(oracle.VSC, wl.coords, wl.spatial_size, [1, 3, 3])
    _, pairs = rb.export()
    np.testing.assert_array_equal(pairs.cpu().numpy(), ref.pairs)
    yo, absb = ref.forward(x, w, b)
    check_features(_to_np(y), yo, absb, RTOL_F32, "pen64")


def test_fullsize_pen_stack_64_grids():
    """VSC 1->32->32->32 on one rule book, then SC 2x2/2, on 64 grids."""
    wl = inputs.make_workload("pen64x64_vsc3x3_sc2")
    size = wl.spatial_size
    ref_v = oracle.Rulebook(oracle.VSC, wl.coords, size, [1, 3, 3])
    rb = spc.build_rulebook(spc.VSC, _t(wl.coords), size, [1, 3, 3])
    _, pairs = rb.export()
    np.testing.assert_array_equal(pairs.cpu().numpy(), ref_v.pairs)
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
    np.testing.assert_array_equal(oc.cpu().numpy(), ref_s.out_coords)
    np.testing.assert_array_equal(pairs.cpu().numpy(), ref_s.pairs)
    yo, absb = ref_s.forward(xo, w, b, x_absb=xa)
    check_features(_to_np(ys), yo, absb, RTOL_F32, "stack SC")


def test_fullsize_encoder_level0_and_downsample():
    """256^3 x 4 surfaces: level-0 VSC (32->32, bf16) and the 2^3 stride-2 SC
    to level 1, rule books exact and sampled rows of both layers."""
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
    np.testing.assert_array_equal(rb.pair_off, ref.pair_off)
    _, pairs = rb.export()
    np.testing.assert_array_equal(pairs.cpu().numpy(), ref.pairs)
    rows = np.sort(np.random.default_rng(1).choice(N, N_SAMPLE_ROWS, replace=False))
    yo, absb = ref.forward_rows(rows, x, w, b, in_dt=oracle.BF16)
    check_features(_to_np(y)[rows], yo, absb, RTOL_BF16, "encoder L0 VSC")
    del ref
    # SC 2^3 stride 2 from the generated input (32 -> 64)
    w2, b2 = make_layer(41, 8, 32, 64, "bf16")
    rbs, ys = _bench_style_layer(spc.SC, wl.coords, size, [1, 2, 2, 2], [1, 2, 2, 2],
                                 _bf16_tensor(x), _bf16_tensor(w2), _t(b2), _lib.BF16, _lib.BF16,
                                 32, 64, torch.bfloat16)
    refs = oracle.Rulebook(oracle.SC, wl.coords, size, [1, 2, 2, 2], [1, 2, 2, 2])
    _say(f"[encoder] oracle SC rule book done, n_out = {refs.n_out}")
    oc, pairs = rbs.export()
    np.testing.assert_array_equal(oc.cpu().numpy(), refs.out_coords)
    np.testing.assert_array_equal(pairs.cpu().numpy(), refs.pairs)
    rows = np.sort(np.random.default_rng(2).choice(refs.n_out, N_SAMPLE_ROWS, replace=False))
    yo, absb = refs.forward_rows(rows, x, w2, b2, in_dt=oracle.BF16)
    check_features(_to_np(ys)[rows], yo, absb, RTOL_BF16, "encoder SC")
