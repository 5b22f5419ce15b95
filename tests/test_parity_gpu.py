"""GPU parity: the HIP library against the oracle, on the same seeded inputs.

Rule books and output site sets must match bit for bit.  Features must meet
both bounds, per element |g - o| <= rtol * S (S = |bias| + sum |x| |w|, the
absolute-sum scale of that output) and normwise ||g - o|| <= rtol ||o||, with
rtol = 1e-5 for fp32 inputs and outputs and 2e-2 when inputs or outputs are
bf16 (fp32 accumulation in every case).
"""
import os
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")

import oracle  # noqa: E402
import paper_1706_01307_amd as spc  # noqa: E402
from paper_1706_01307_amd import inputs  # noqa: E402
from tests import dense_ref  # noqa: E402
from tests.rb_check import check_rulebook  # noqa: E402

pytestmark = pytest.mark.gpu

RTOL_F32 = 1e-5
RTOL_BF16 = 2e-2


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.init()


def _t(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _bf16_tensor(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).cuda()


def _to_np(t):
    if t.dtype == torch.bfloat16:
        return inputs.bf16_bits_to_f32(t.view(torch.int16).cpu().numpy().view(np.uint16))
    return t.cpu().numpy()


def check_features(g, o, absb, rtol, what=""):
    g = g.astype(np.float64)
    err = np.abs(g - o)
    bad = err > rtol * absb
    assert not bad.any(), (
        f"{what}: {int(bad.sum())} elements over the bound; worst "
        f"{float((err / np.maximum(absb, 1e-300)).max()):.3e}")
    no = np.linalg.norm(o)
    if no > 0:
        assert np.linalg.norm(g - o) <= rtol * no, what


def make_layer(rng_seed, K, C_in, C_out, dtype, with_bias=True):
    w = inputs.normal_f32((K, C_in, C_out), std=1.0 / np.sqrt(K * C_in), seed=rng_seed)
    b = inputs.normal_f32((C_out,), std=0.1, seed=rng_seed + 1) if with_bias else None
    if dtype == "bf16":
        return inputs.to_bf16_bits(w), b
    return w, b


def run_layer(kind, coords, size, f, s, x, w, b, dtype, out_dtype, sync=True):
    """GPU rule book + forward; returns (out_coords, pairs, pair_off, y as float)."""
    tc = _t(coords)
    rb = spc.build_rulebook(kind, tc, size, f, s, sync=sync)
    if not sync:
        assert rb.status() == spc.OK
    if dtype == "bf16":
        xt, wt = _bf16_tensor(x), _bf16_tensor(w)
    else:
        xt, wt = _t(x), _t(w)
    bt = None if b is None else _t(b)
    od = torch.bfloat16 if out_dtype == "bf16" else torch.float32
    fwd = spc.vsc_forward if kind == spc.VSC else spc.sc_forward
    y = fwd(rb, xt, wt, bt, out_dtype=od)
    oc, pairs = rb.export()
    torch.cuda.synchronize()
    return oc.cpu().numpy(), pairs.cpu().numpy(), rb.pair_off, _to_np(y), rb


def compare_layer(kind, coords, size, f, s, C_in, C_out, dtype="f32", out_dtype=None,
                  seed=0, with_bias=True, x=None, what=""):
    out_dtype = out_dtype or dtype
    K = int(np.prod(f))
    if x is None:
        xf = inputs.normal_f32((len(coords), C_in), seed=seed)
        x = inputs.to_bf16_bits(xf) if dtype == "bf16" else xf
    w, b = make_layer(seed + 100, K, C_in, C_out, dtype, with_bias)
    _say(f"[{what}] kind={kind} N={len(coords)} size={list(size)} f={list(f)} s={list(s)} "
         f"C={C_in}->{C_out} {dtype}->{out_dtype}")
    oc, pairs, pair_off, y, rb = run_layer(kind, coords, size, f, s, x, w, b, dtype, out_dtype)
    ref = oracle.Rulebook(kind, coords, size, f, s)
    check_rulebook(oc, pairs, pair_off, ref)
    yo, absb = ref.forward(x, w, b, in_dt=oracle.BF16 if dtype == "bf16" else oracle.F32)
    rtol = RTOL_F32 if (dtype == "f32" and out_dtype == "f32") else RTOL_BF16
    check_features(y, yo, absb, rtol, what)
    return y, yo, absb, ref, rb


# ---------------------------------------------------------------------------
# Workload-shaped cases at oracle-friendly sizes (several tiles + ragged tail)
# ---------------------------------------------------------------------------

def test_pen_vsc_c1_to_16_f32():
    """One 64x64 pen-stroke grid, VSC 3x3, 1 -> 16 planes, fp32 (input 1.0)."""
    coords = inputs.pen_strokes(1, 64, seed=0, target=400)
    x = np.ones((len(coords), 1), np.float32)
    compare_layer(spc.VSC, coords, [1, 64, 64], [1, 3, 3], [1, 1, 1], 1, 16, x=x,
                  what="pen64 c1x16")


def test_pen_stack_vsc_vsc_vsc_sc_f32():
    """Pen grids: VSC 1->32, 32->32, 32->32 on one rule book, then SC 2x2/2."""
    coords = inputs.pen_strokes(8, 64, seed=1, target=400)
    size = [8, 64, 64]
    ref_vsc = oracle.Rulebook(oracle.VSC, coords, size, [1, 3, 3])
    rb = spc.build_rulebook(spc.VSC, _t(coords), size, [1, 3, 3])
    x = np.ones((len(coords), 1), np.float32)
    xg = _t(x)
    xo, xa = x.astype(np.float64), np.abs(x).astype(np.float64)
    chans = [(1, 32), (32, 32), (32, 32)]
    for li, (ci, co) in enumerate(chans):
        w, b = make_layer(10 + li, 9, ci, co, "f32")
        xg = spc.vsc_forward(rb, xg, _t(w), _t(b))
        # oracle: its own previous (rounded to fp32) output as input
        yo, absb = ref_vsc.forward(oracle.round_to(xo, oracle.F32) if li else x, w, b,
                                   x_absb=xa)
        check_features(_to_np(xg), yo, absb, RTOL_F32, f"stack layer {li}")
        xo, xa = yo, absb
    w, b = make_layer(20, 4, 32, 32, "f32")
    rbs = spc.build_rulebook(spc.SC, _t(coords), size, [1, 2, 2], [1, 2, 2])
    ys = spc.sc_forward(rbs, xg, _t(w), _t(b))
    ref_sc = oracle.Rulebook(oracle.SC, coords, size, [1, 2, 2], [1, 2, 2])
    oc, pairs = rbs.export()
    check_rulebook(oc.cpu().numpy(), pairs.cpu().numpy(), rbs.pair_off, ref_sc)
    yo, absb = ref_sc.forward(oracle.round_to(xo, oracle.F32), w, b, x_absb=xa)
    check_features(_to_np(ys), yo, absb, RTOL_F32, "stack SC")


def test_surface_vsc3_c32_f32():
    coords = inputs.surfaces(2, 48, 6.0, 20.0, seed=5, target=6000)
    compare_layer(spc.VSC, coords, [2, 48, 48, 48], [1, 3, 3, 3], [1, 1, 1, 1], 32, 32,
                  what="surf48 c32 f32")


@pytest.mark.parametrize("out_dtype", ["bf16", "f32"])
def test_surface_vsc3_c64_bf16(out_dtype):
    coords = inputs.surfaces(2, 64, 8.0, 30.0, seed=6, target=9000)
    compare_layer(spc.VSC, coords, [2, 64, 64, 64], [1, 3, 3, 3], [1, 1, 1, 1], 64, 64,
                  dtype="bf16", out_dtype=out_dtype, what="surf64 c64 bf16")


@pytest.mark.parametrize("ci,co", [(32, 64), (64, 96), (96, 96), (128, 128), (32, 32)])
def test_encoder_widths_bf16(ci, co):
    """Channel widths of the four-level encoder: VSC and SC 2^3 stride 2."""
    coords = inputs.surfaces(1, 48, 6.0, 20.0, seed=7, target=5000)
    size = [1, 48, 48, 48]
    compare_layer(spc.VSC, coords, size, [1, 3, 3, 3], [1, 1, 1, 1], ci, co, dtype="bf16",
                  what=f"vsc {ci}->{co}")
    compare_layer(spc.SC, coords, size, [1, 2, 2, 2], [1, 2, 2, 2], ci, co, dtype="bf16",
                  what=f"sc {ci}->{co}")


@pytest.mark.parametrize("ci,co", [(16, 16), (64, 32), (96, 48), (128, 64)])
def test_f32_mfma_widths(ci, co):
    coords = inputs.surfaces(1, 40, 5.0, 16.0, seed=8, target=3000)
    compare_layer(spc.VSC, coords, [1, 40, 40, 40], [1, 3, 3, 3], [1, 1, 1, 1], ci, co,
                  what=f"f32 {ci}->{co}")


# ---------------------------------------------------------------------------
# Edge cases
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("kind", [0, 1])
def test_empty_input(kind):
    coords = np.zeros((0, 3), np.int32)
    f = [1, 3, 3] if kind == spc.VSC else [1, 2, 2]
    s = [1, 1, 1] if kind == spc.VSC else [1, 2, 2]
    rb = spc.build_rulebook(kind, _t(coords), [1, 8, 8], f, s)
    assert rb.n_out == 0 and rb.pair_off[-1] == 0
    y = (spc.vsc_forward if kind == spc.VSC else spc.sc_forward)(
        rb, _t(np.zeros((0, 4), np.float32)), _t(np.ones((rb.K, 4, 4), np.float32)))
    assert y.shape == (0, 4)


def test_single_site_and_isolated_sites():
    compare_layer(spc.VSC, np.array([[0, 3, 4]], np.int32), [1, 8, 8], [1, 3, 3], [1, 1, 1],
                  4, 4, what="N=1")
    # every other site on a lattice of spacing 2: no site has a neighbour
    c = np.argwhere(np.ones((2, 16, 16), bool)[:, ::2, ::2]).astype(np.int32)
    c[:, 1:] *= 2
    compare_layer(spc.VSC, c, [2, 16, 16], [1, 3, 3], [1, 1, 1], 32, 32, what="isolated")


def test_fully_dense_cube():
    c = np.argwhere(np.ones((2, 12, 12, 12), bool)).astype(np.int32)
    compare_layer(spc.VSC, c, [2, 12, 12, 12], [1, 3, 3, 3], [1, 1, 1, 1], 32, 32,
                  dtype="bf16", what="dense cube")
    compare_layer(spc.SC, c, [2, 12, 12, 12], [1, 3, 3, 3], [1, 2, 2, 2], 16, 16,
                  what="dense cube SC 3/2")


@pytest.mark.parametrize("ci,co", [(3, 5), (1, 1), (7, 33), (20, 17), (33, 16)])
def test_ragged_channels_vector_path(ci, co):
    coords = inputs.surfaces(1, 24, 3.0, 10.0, seed=9, target=1500)
    compare_layer(spc.VSC, coords, [1, 24, 24, 24], [1, 3, 3, 3], [1, 1, 1, 1], ci, co,
                  what=f"ragged {ci}->{co}")
    compare_layer(spc.VSC, coords, [1, 24, 24, 24], [1, 3, 3, 3], [1, 1, 1, 1], ci, co,
                  dtype="bf16", what=f"ragged bf16 {ci}->{co}")


def test_vector_path_forced_on_mfma_shapes(monkeypatch):
    monkeypatch.setenv("SPCONV_FORCE_PATH", "vec")
    coords = inputs.surfaces(1, 32, 4.0, 12.0, seed=10, target=2500)
    compare_layer(spc.VSC, coords, [1, 32, 32, 32], [1, 3, 3, 3], [1, 1, 1, 1], 64, 64,
                  dtype="bf16", what="forced vec bf16")
    compare_layer(spc.VSC, coords, [1, 32, 32, 32], [1, 3, 3, 3], [1, 1, 1, 1], 32, 32,
                  what="forced vec f32")


@pytest.mark.parametrize("f,s", [([1, 1, 7], [1, 1, 1]), ([1, 7, 1], [1, 1, 1]),
                                 ([1, 5, 5], [1, 1, 1]), ([1, 1, 1], [1, 1, 1])])
def test_vsc_filter_shapes(f, s):
    coords = inputs.pen_strokes(3, 40, seed=12, target=200)
    compare_layer(spc.VSC, coords, [3, 40, 40], f, s, 16, 16, what=f"vsc f={f}")


@pytest.mark.parametrize("f,s", [([1, 3, 3], [1, 2, 2]), ([1, 2, 2], [1, 2, 2]),
                                 ([1, 3, 3], [1, 1, 1]), ([1, 1, 1], [1, 2, 2]),
                                 ([1, 4, 2], [1, 3, 1])])
def test_sc_filter_shapes(f, s):
    coords = inputs.pen_strokes(3, 41, seed=13, target=250)
    compare_layer(spc.SC, coords, [3, 41, 41], f, s, 16, 32, what=f"sc f={f} s={s}")


def test_vsc_5cube_many_offsets():
    coords = inputs.surfaces(1, 24, 3.0, 10.0, seed=14, target=1500)
    compare_layer(spc.VSC, coords, [1, 24, 24, 24], [1, 5, 5, 5], [1, 1, 1, 1], 32, 32,
                  dtype="bf16", what="5^3")


def test_d1_and_odd_extents():
    rng = np.random.default_rng(15)
    c = dense_ref.random_sites(rng, [3, 1000], 0.3)
    compare_layer(spc.VSC, c, [3, 1000], [1, 3], [1, 1], 16, 16, what="1-d vsc")
    compare_layer(spc.SC, c, [3, 1000], [1, 3], [1, 2], 16, 16, what="1-d sc")
    c = dense_ref.random_sites(rng, [2, 63, 63], 0.1)
    compare_layer(spc.SC, c, [2, 63, 63], [1, 3, 3], [1, 2, 2], 32, 32, what="63->31")


def test_wide_hash_layout():
    """Keys wider than 64 - row bits use the two-array table layout."""
    rng = np.random.default_rng(16)
    n = 3000
    c = np.stack([rng.integers(0, 60000, n), rng.integers(0, 60000, n),
                  rng.integers(0, 60000, n), rng.integers(0, 60000, n)], 1).astype(np.int32)
    c = np.unique(c, axis=0)
    # add neighbours so that the rule book is not trivial
    c = np.unique(np.concatenate([c, c + [0, 0, 0, 1], c + [0, 1, 0, 0]]), axis=0)
    c = c[np.all(c < 60000, axis=1)].astype(np.int32)
    compare_layer(spc.VSC, c, [60000] * 4, [1, 3, 3, 3], [1, 1, 1, 1], 16, 16,
                  what="wide keys")


RULEBOOK_CASES = [
    # kind, grid, f, s, C_in, C_out, dtype
    (0, "surf", [1, 3, 3, 3], [1, 1, 1, 1], 64, 64, "bf16"),
    (1, "surf", [1, 2, 2, 2], [1, 2, 2, 2], 32, 64, "f32"),
    (1, "surf", [1, 3, 3, 3], [1, 2, 2, 2], 16, 32, "f32"),
    (0, "pen", [1, 3, 3], [1, 1, 1], 16, 16, "f32"),
    (1, "pen", [1, 3, 3], [1, 2, 2], 16, 16, "f32"),
    (0, "aniso", [1, 3, 5, 1], [1, 1, 1, 1], 16, 16, "f32"),
    (1, "aniso", [1, 2, 3, 1], [1, 2, 1, 1], 16, 16, "f32"),
]


def _rulebook_case_sites(name):
    if name == "surf":
        return inputs.surfaces(2, 37, 4.0, 14.0, seed=31, target=2500), [2, 37, 37, 37]
    if name == "pen":
        return inputs.pen_strokes(5, 45, seed=32, target=300), [5, 45, 45]
    rng = np.random.default_rng(33)
    size = [3, 5, 70, 3]
    return dense_ref.random_sites(rng, size, 0.3), size


@pytest.mark.parametrize("path", ["hash", "table", "grid", "grid3"])
@pytest.mark.parametrize("case", range(len(RULEBOOK_CASES)))
def test_rulebook_paths(monkeypatch, path, case):
    """Hashed and dense-grid rule books give the same (oracle) result: hash
    = the sorted-brick map for VSC (the site table for SC), table = the
    open-addressing table of sites for both; grid3 ranks a small grid's cells
    with the three-launch multi-block path instead of one workgroup."""
    monkeypatch.setenv("SPCONV_RULEBOOK", path)
    kind, name, f, s, ci, co, dt = RULEBOOK_CASES[case]
    coords, size = _rulebook_case_sites(name)
    compare_layer(kind, coords, size, f, s, ci, co, dtype=dt, what=f"{path} {name}")


def test_grid_forced_on_sparse_wide_grid(monkeypatch):
    """The dense grid also serves grids far larger than the site count."""
    monkeypatch.setenv("SPCONV_RULEBOOK", "grid")
    rng = np.random.default_rng(34)
    c = np.unique(rng.integers(0, [2, 1500, 1500], size=(4000, 3)), axis=0).astype(np.int32)
    c = np.unique(np.concatenate([c, c + [0, 0, 1], c + [0, 1, 1]]), axis=0)
    c = c[np.all(c < [2, 1500, 1500], axis=1)].astype(np.int32)
    compare_layer(spc.VSC, c, [2, 1500, 1500], [1, 3, 3], [1, 1, 1], 16, 16, what="grid sparse")
    compare_layer(spc.SC, c, [2, 1500, 1500], [1, 3, 3], [1, 2, 2], 16, 16,
                  what="grid sparse SC")


@pytest.mark.parametrize("f", [3, 5])
def test_brick_map_on_grids_too_large_for_the_dense_grid(f):
    """Grids of 2^31 cells (no dense grid): VSC takes the sorted-brick map by
    default; surfaces cut from a huge volume, sparse scattered sites and
    sites on the grid's faces and corners (bricks whose neighbours fall off
    the grid), against the oracle."""
    rng = np.random.default_rng(35 + f)
    size = [2, 4096, 2048, 128]
    shell = inputs.surfaces(2, 64, 6.0, 28.0, seed=40 + f, target=4000)
    shell = shell + np.array([0, 4000, 100, 60], np.int32)          # near a far face
    scattered = np.unique(rng.integers(0, size, size=(3000, 4)), axis=0)
    corners = np.array([[b, x, y, z] for b in (0, 1) for x in (0, 1, 4094, 4095)
                        for y in (0, 2047) for z in (0, 1, 126, 127)], np.int64)
    c = np.unique(np.concatenate([shell, scattered, corners]), axis=0)
    c = c[np.all((c >= 0) & (c < size), axis=1)].astype(np.int32)
    _say(f"[brick map] f={f} N={len(c)}")
    compare_layer(spc.VSC, c, size, [1, f, f, f], [1, 1, 1, 1], 16, 16, what=f"brick map f{f}")


def test_permuted_rows():
    """VSC output permutes with its input; SC output does not move."""
    coords = inputs.pen_strokes(4, 32, seed=17, target=150)
    size = [4, 32, 32]
    x = inputs.normal_f32((len(coords), 16), seed=3)
    w, b = make_layer(5, 9, 16, 16, "f32")
    perm = np.random.default_rng(0).permutation(len(coords))
    _, _, _, y0, _ = run_layer(spc.VSC, coords, size, [1, 3, 3], [1, 1, 1], x, w, b, "f32", "f32")
    _, _, _, y1, _ = run_layer(spc.VSC, coords[perm], size, [1, 3, 3], [1, 1, 1], x[perm], w, b,
                               "f32", "f32")
    np.testing.assert_array_equal(y1, y0[perm])
    w2, b2 = make_layer(6, 4, 16, 16, "f32")
    oc0, _, _, s0, _ = run_layer(spc.SC, coords, size, [1, 2, 2], [1, 2, 2], x, w2, b2, "f32",
                                 "f32")
    oc1, _, _, s1, _ = run_layer(spc.SC, coords[perm], size, [1, 2, 2], [1, 2, 2], x[perm], w2,
                                 b2, "f32", "f32")
    np.testing.assert_array_equal(oc0, oc1)
    np.testing.assert_allclose(s0, s1, rtol=1e-6, atol=1e-6)


def test_repeated_runs_bitwise_identical():
    coords = inputs.surfaces(1, 48, 6.0, 20.0, seed=18, target=5000)
    size = [1, 48, 48, 48]
    xb = inputs.to_bf16_bits(inputs.normal_f32((len(coords), 64), seed=1))
    w, b = make_layer(7, 27, 64, 64, "bf16")
    outs = []
    for _ in range(3):
        oc, pairs, _, y, _ = run_layer(spc.VSC, coords, size, [1, 3, 3, 3], [1, 1, 1, 1], xb, w,
                                       b, "bf16", "f32")
        outs.append((pairs, y))
    for p, y in outs[1:]:
        np.testing.assert_array_equal(p, outs[0][0])
        np.testing.assert_array_equal(y, outs[0][1])


def test_async_build_and_reuse():
    coords = inputs.surfaces(1, 32, 4.0, 12.0, seed=19, target=2000)
    size = [1, 32, 32, 32]
    x = inputs.normal_f32((len(coords), 32), seed=2)
    w, b = make_layer(8, 27, 32, 32, "f32")
    oc, pairs, pair_off, y, rb = run_layer(spc.VSC, coords, size, [1, 3, 3, 3], [1, 1, 1, 1],
                                           x, w, b, "f32", "f32", sync=False)
    ref = oracle.Rulebook(oracle.VSC, coords, size, [1, 3, 3, 3])
    check_rulebook(oc, pairs, pair_off, ref)
    # the same rule book serves a second layer
    w2, b2 = make_layer(9, 27, 32, 32, "f32")
    y2 = spc.vsc_forward(rb, _t(x), _t(w2), _t(b2))
    yo, absb = ref.forward(x, w2, b2)
    check_features(_to_np(y2), yo, absb, RTOL_F32, "reuse")


# ---------------------------------------------------------------------------
# Device-detected errors
# ---------------------------------------------------------------------------

def _status(kind, coords, size, f, s):
    try:
        spc.build_rulebook(kind, _t(coords), size, f, s)
        return spc.OK
    except spc.SpconvError as e:
        return e.status


@pytest.mark.parametrize("path", ["hash", "table", "grid"])
@pytest.mark.parametrize("kind", [0, 1])
def test_errors_match_oracle(monkeypatch, kind, path):
    monkeypatch.setenv("SPCONV_RULEBOOK", path)
    f = [1, 3, 3] if kind == spc.VSC else [1, 2, 2]
    s = [1, 1, 1] if kind == spc.VSC else [1, 2, 2]
    dup = np.array([[0, 1, 1], [0, 2, 2], [0, 1, 1]], np.int32)
    oor = np.array([[0, 1, 1], [0, 8, 2]], np.int32)
    neg = np.array([[0, 1, -1]], np.int32)
    bad_b = np.array([[2, 1, 1]], np.int32)
    for c in (dup, oor, neg, bad_b):
        assert _status(kind, c, [2, 8, 8], f, s) == oracle.status_of_build(kind, c, [2, 8, 8],
                                                                           f, s)
    assert _status(kind, dup, [2, 8, 8], f, s) == spc.EDUP
    assert _status(kind, oor, [2, 8, 8], f, s) == spc.ERANGE


@pytest.mark.parametrize("path", ["hash", "grid"])
def test_async_error_reported_by_status(monkeypatch, path):
    monkeypatch.setenv("SPCONV_RULEBOOK", path)
    dup = np.array([[0, 1, 1], [0, 1, 1]], np.int32)
    rb = spc.build_rulebook(spc.VSC, _t(dup), [1, 8, 8], [1, 3, 3], sync=False)
    assert rb.status() == spc.EDUP
    rb.close()
    oor = np.array([[0, 1, 1], [0, 1, 9]], np.int32)
    rb = spc.build_rulebook(spc.SC, _t(oor), [1, 8, 8], [1, 2, 2], [1, 2, 2], sync=False)
    assert rb.status() == spc.ERANGE
    rb.close()


def test_table_full_is_reported_not_hung(monkeypatch):
    monkeypatch.setenv("SPCONV_RULEBOOK", "hash")
    monkeypatch.setenv("SPCONV_TEST_HASH_SLOTS", "8")
    coords = inputs.pen_strokes(1, 32, seed=20, target=100)
    assert len(coords) > 8
    assert _status(spc.VSC, coords, [1, 32, 32], [1, 3, 3], [1, 1, 1]) == spc.ECAP
    monkeypatch.setenv("SPCONV_TEST_HASH_SLOTS", str(len(coords)))
    # a table exactly as large as the site set still works (full buckets)
    compare_layer(spc.VSC, coords, [1, 32, 32], [1, 3, 3], [1, 1, 1], 16, 16, what="tight table")


def test_kind_mismatch():
    coords = inputs.pen_strokes(1, 16, seed=21, target=30)
    rb = spc.build_rulebook(spc.VSC, _t(coords), [1, 16, 16], [1, 3, 3])
    from paper_1706_01307_amd import _lib
    lib = _lib.load()
    x = _t(np.zeros((len(coords), 4), np.float32))
    w = _t(np.zeros((9, 4, 4), np.float32))
    y = _t(np.zeros((len(coords), 4), np.float32))
    st = lib.spconv_sc_forward(rb.handle, 0, x.data_ptr(), w.data_ptr(), None, 0, y.data_ptr(),
                               4, 4, None)
    assert st == spc.EINVAL


def test_non_contiguous_coords_through_python_api():
    """Column-major coordinate tensors are made contiguous before the ABI."""
    coords = inputs.pen_strokes(2, 32, seed=22, target=120)
    cf = torch.from_numpy(np.asfortranarray(coords)).cuda()
    assert not cf.is_contiguous()
    rb = spc.build_rulebook(spc.VSC, cf, [2, 32, 32], [1, 3, 3])
    ref = oracle.Rulebook(oracle.VSC, coords, [2, 32, 32], [1, 3, 3])
    oc, pairs = rb.export()
    check_rulebook(oc.cpu().numpy(), pairs.cpu().numpy(), rb.pair_off, ref)


@pytest.mark.parametrize("path", ["mfma", "vec"])
def test_matrix_core_shapes_both_paths(monkeypatch, path):
    """Matrix-core shapes, through the matrix-core kernel and the vector path
    (SPCONV_FORCE_PATH=vec): wide outputs walk column chunks; SC layers,
    generic filter sizes and f = 1 included."""
    if path == "vec":
        monkeypatch.setenv("SPCONV_FORCE_PATH", "vec")
    coords = inputs.surfaces(2, 40, 5.0, 16.0, seed=24, target=4000)
    size = [2, 40, 40, 40]
    compare_layer(spc.VSC, coords, size, [1, 3, 3, 3], [1, 1, 1, 1], 64, 128,
                  dtype="bf16", what=f"{path} C_out 128")
    compare_layer(spc.VSC, coords, size, [1, 3, 3, 3], [1, 1, 1, 1], 32, 64,
                  what=f"{path} f32")
    compare_layer(spc.VSC, coords, size, [1, 3, 3, 3], [1, 1, 1, 1], 64, 64,
                  dtype="bf16", out_dtype="f32", what=f"{path} bf16->f32")
    compare_layer(spc.VSC, coords, size, [1, 1, 3, 3], [1, 1, 1, 1], 64, 64,
                  dtype="bf16", what=f"{path} 1x3x3")
    compare_layer(spc.VSC, coords, size, [1, 5, 5, 5], [1, 1, 1, 1], 64, 64,
                  dtype="bf16", what=f"{path} 5^3")
    compare_layer(spc.VSC, coords, size, [1, 1, 1, 1], [1, 1, 1, 1], 32, 64,
                  what=f"{path} f=1")
    compare_layer(spc.SC, coords, size, [1, 2, 2, 2], [1, 2, 2, 2], 64, 64,
                  dtype="bf16", what=f"{path} SC 2/2")
    compare_layer(spc.SC, coords, size, [1, 3, 3, 3], [1, 2, 2, 2], 32, 128,
                  what=f"{path} SC 3/2 f32")


@pytest.mark.parametrize("path", ["hash", "grid"])
def test_forward_on_both_rulebook_paths(monkeypatch, path):
    """The forward walks the schedule and gather map of either rule-book
    path."""
    monkeypatch.setenv("SPCONV_RULEBOOK", path)
    coords = inputs.surfaces(3, 36, 4.0, 14.0, seed=25, target=3000)
    compare_layer(spc.VSC, coords, [3, 36, 36, 36], [1, 3, 3, 3], [1, 1, 1, 1], 64, 64,
                  dtype="bf16", what=f"forward {path}")
    compare_layer(spc.SC, coords, [3, 36, 36, 36], [1, 2, 2, 2], [1, 2, 2, 2], 64, 64,
                  dtype="bf16", what=f"forward SC {path}")


# Grids that exercise the grouped probes (VSC 3^3 and SC 2^3 stride 2 on 4-D
# grids read 16-byte cell groups) at their edges: odd and tiny extents, and
# extents of 1 that send a build to the one-cell-per-load probe instead.
GROUP_PROBE_SIZES = [[2, 3, 5, 7], [1, 2, 2, 2], [3, 9, 2, 4], [2, 6, 6, 1], [2, 1, 5, 5],
                     [1, 17, 3, 33]]


@pytest.mark.parametrize("density", [0.5, 0.06])
@pytest.mark.parametrize("size", GROUP_PROBE_SIZES)
def test_group_probe_edges(monkeypatch, size, density):
    monkeypatch.setenv("SPCONV_RULEBOOK", "grid")
    rng = np.random.default_rng(int(np.prod(size)) + int(density * 100))
    c = dense_ref.random_sites(rng, size, density)
    if len(c) == 0:
        c = np.zeros((1, 4), np.int32)
    compare_layer(spc.VSC, c, size, [1, 3, 3, 3], [1, 1, 1, 1], 32, 32, dtype="bf16",
                  what="group probe VSC")
    if all(v >= 2 for v in size[1:]):
        compare_layer(spc.SC, c, size, [1, 2, 2, 2], [1, 2, 2, 2], 32, 32, dtype="bf16",
                      what="group probe SC")
