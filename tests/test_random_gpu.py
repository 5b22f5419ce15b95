"""Seeded random layers against the oracle: grid extents (odd, tiny, with
extent 1, mixed), filter shapes and strides, site densities, channel counts
on both sides of the matrix-core shapes, dtypes and both site maps.  Each
case: rule book (output sites, pair offsets, pairs) bit for bit, forward
within the parity bounds."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

import paper_1706_01307_amd as spc  # noqa: E402
from tests import dense_ref  # noqa: E402
from tests.test_parity_gpu import _say, compare_layer  # noqa: E402

pytestmark = pytest.mark.gpu

CHANNELS = [(1, 16), (16, 16), (32, 32), (32, 64), (64, 64), (64, 32), (96, 96), (128, 128),
            (7, 33), (48, 16)]


def _case(seed):
    rng = np.random.default_rng(1000 + seed)
    D = int(rng.integers(2, 5))
    kind = int(rng.integers(0, 2))
    size = [int(rng.integers(1, 4))] + [int(rng.choice([1, 2, 3, 5, 8, 13, 16, 31, 64]))
                                       for _ in range(D - 1)]
    if kind == spc.VSC:
        f = [1] + [int(rng.choice([1, 3, 3, 3, 5])) for _ in range(D - 1)]
        s = [1] * D
    else:
        f = [1] + [int(rng.integers(1, 4)) for _ in range(D - 1)]
        s = [1] + [int(rng.integers(1, 4)) for _ in range(D - 1)]
        f = [min(fj, max(sz, 1)) for fj, sz in zip(f, size)]
    density = float(rng.choice([0.02, 0.1, 0.3, 0.7, 1.0]))
    ci, co = CHANNELS[int(rng.integers(0, len(CHANNELS)))]
    dtype = "bf16" if (ci % 32 == 0 and rng.random() < 0.5) else "f32"
    out_dtype = dtype if rng.random() < 0.7 else ("f32" if dtype == "bf16" else "bf16")
    path = str(rng.choice(["grid", "hash", "grid3", "table"]))
    c = dense_ref.random_sites(rng, size, density)
    if len(c) == 0:          # (empty inputs have their own test)
        c = np.array([[int(rng.integers(0, e)) for e in size]], np.int32)
    # keep the oracle's double-precision forward to a second or so
    while len(c) > 1 and len(c) * int(np.prod(f)) * ci * co > 3e8:
        c = c[::2]
    return kind, c, size, f, s, ci, co, dtype, out_dtype, path


@pytest.mark.parametrize("seed", range(128))
def test_random_layer(monkeypatch, seed):
    kind, c, size, f, s, ci, co, dtype, out_dtype, path = _case(seed)
    monkeypatch.setenv("SPCONV_RULEBOOK", path)
    _say(f"[random {seed}] path={path}")
    compare_layer(kind, c, size, f, s, ci, co, dtype=dtype, out_dtype=out_dtype, seed=seed,
                  what=f"random {seed}")


@pytest.mark.parametrize("seed", range(48))
def test_random_fused_forward(seed):
    """The forward with a random subset of the block epilogue (scale, shift,
    residual, ReLU) fused, on random layers."""
    import oracle
    from paper_1706_01307_amd import inputs
    from tests.test_ops_gpu import _dev, _feats, _odt
    from tests.test_parity_gpu import RTOL_BF16, RTOL_F32, _t, _to_np, check_features
    kind, c, size, f, s, ci, co, dtype, out_dtype, path = _case(seed + 500)
    rng = np.random.default_rng(seed)
    use_s, use_b, use_r, relu = (bool(v) for v in rng.integers(0, 2, size=4))
    rb = spc.build_rulebook(kind, _t(c), size, f, s)
    ref = oracle.Rulebook(kind, c, size, f, s)
    K = ref.K
    x = _feats(len(c), ci, dtype, 11 * seed + 1)
    wf = inputs.normal_f32((K, ci, co), std=1.0 / np.sqrt(K * ci), seed=11 * seed + 2)
    w = inputs.to_bf16_bits(wf) if dtype == "bf16" else wf
    scale = inputs.normal_f32((co,), std=1.0, seed=11 * seed + 3)
    shift = inputs.normal_f32((co,), std=0.5, seed=11 * seed + 4)
    res = _feats(ref.n_out, co, out_dtype, 11 * seed + 5)
    _say(f"[random fused {seed}] kind={kind} N={len(c)} f={f} s={s} C={ci}->{co} {dtype}->"
         f"{out_dtype} parts={use_s, use_b, use_r, relu}")
    odt = torch.bfloat16 if out_dtype == "bf16" else torch.float32
    y = spc.forward_fused(rb, _dev(x, dtype), _dev(w, dtype),
                          scale=_t(scale) if use_s else None, shift=_t(shift) if use_b else None,
                          residual=_dev(res, out_dtype) if use_r else None, relu=relu,
                          out_dtype=odt)
    y64, absb = ref.forward(x, w, None, in_dt=_odt(dtype))
    zo, bound = oracle.fused_epilogue(y64, absb, scale if use_s else None,
                                      shift if use_b else None, res if use_r else None,
                                      relu, _odt(out_dtype))
    rtol = RTOL_F32 if dtype == "f32" and out_dtype == "f32" else RTOL_BF16
    check_features(_to_np(y), zo, bound, rtol, "fused")


@pytest.mark.parametrize("seed", range(40))
def test_random_small_vsc_build(monkeypatch, seed):
    """The one-workgroup build of small VSC layers (SPCONV_RULEBOOK=small):
    random extents, filters 1/3/5 per dimension, densities and channel
    counts, at most 2048 sites on at most 2^18 cells of 2^B per dimension,
    2^B >= extent + (f - 1) / 2 (the workgroup's capacity: 3 samples of
    29^3, of 200^2), against the oracle (rule book bit for bit, forward
    within the parity bounds)."""
    rng = np.random.default_rng(5000 + seed)
    D = int(rng.integers(2, 5))
    ext = [1, 2, 3, 7, 16, 29] + ([64, 200] if D < 4 else [])
    size = [int(rng.integers(1, 4))] + [int(rng.choice(ext)) for _ in range(D - 1)]
    f = [1] + [int(rng.choice([1, 3, 3, 5])) for _ in range(D - 1)]
    c = dense_ref.random_sites(rng, size, float(rng.choice([0.01, 0.1, 0.5, 1.0])))
    if len(c) == 0:
        c = np.array([[int(rng.integers(0, e)) for e in size]], np.int32)
    if len(c) > 2048:
        c = c[np.sort(rng.choice(len(c), 2048, replace=False))]
    ci, co = CHANNELS[int(rng.integers(0, len(CHANNELS)))]
    dtype = "bf16" if (ci % 32 == 0 and rng.random() < 0.5) else "f32"
    monkeypatch.setenv("SPCONV_RULEBOOK", "small")
    _say(f"[small {seed}] N={len(c)}")
    compare_layer(spc.VSC, c, size, f, [1] * D, ci, co, dtype=dtype, seed=seed,
                  what=f"small {seed}")


def test_small_build_errors_and_boundary(monkeypatch):
    """Duplicates and out-of-range sites through the small build, and a layer
    of exactly 2048 sites (the largest it takes) next to one of 2049 (which
    takes the grid path)."""
    from tests.test_parity_gpu import _t
    import oracle
    monkeypatch.setenv("SPCONV_RULEBOOK", "small")
    dup = np.array([[0, 3, 4], [0, 5, 5], [0, 3, 4]], np.int32)
    with pytest.raises(spc.SpconvError) as e:
        spc.build_rulebook(spc.VSC, _t(dup), [1, 8, 8], [1, 3, 3])
    assert e.value.status == spc.EDUP
    oor = np.array([[0, 3, 4], [0, 8, 5]], np.int32)
    with pytest.raises(spc.SpconvError) as e:
        spc.build_rulebook(spc.VSC, _t(oor), [1, 8, 8], [1, 3, 3])
    assert e.value.status == spc.ERANGE == oracle.status_of_build(oracle.VSC, oor, [1, 8, 8],
                                                                   [1, 3, 3])
    rng = np.random.default_rng(3)
    full = dense_ref.random_sites(rng, [2, 64, 64], 0.5)
    for n in (2048, 2049):
        c = full[np.sort(rng.choice(len(full), n, replace=False))]
        compare_layer(spc.VSC, c, [2, 64, 64], [1, 3, 3], [1, 1, 1], 16, 16, seed=n,
                      what=f"boundary {n}")


@pytest.mark.parametrize("seed", range(12))
def test_random_few_input_planes(seed):
    """Layers of 1-4 input planes and 16/32/48 output planes on at least
    2048 input sites (where the output count is as large: the
    one-lane-per-16-columns kernel), f32 and bf16, VSC and SC, against the
    oracle."""
    rng = np.random.default_rng(7000 + seed)
    D = int(rng.integers(3, 5))
    kind = int(rng.integers(0, 2))
    ext = [24, 31, 40] if D == 4 else [64, 80, 96]
    size = [int(rng.integers(1, 3))] + [int(rng.choice(ext)) for _ in range(D - 1)]
    if kind == spc.VSC:
        f, s = [1] + [3] * (D - 1), [1] * D
    else:
        f, s = [1] + [2] * (D - 1), [1] + [int(rng.choice([1, 2]))] * (D - 1)
    c = dense_ref.random_sites(rng, size, 0.5 if D == 3 else 0.08)
    ci = int(rng.integers(1, 5))
    co = int(rng.choice([16, 32, 48]))
    dtype = "bf16" if rng.random() < 0.5 else "f32"
    out_dtype = dtype if rng.random() < 0.5 else ("f32" if dtype == "bf16" else "bf16")
    _say(f"[few planes {seed}] N={len(c)}")
    assert len(c) >= 2048
    compare_layer(kind, c, size, f, s, ci, co, dtype=dtype, out_dtype=out_dtype, seed=seed,
                  what=f"few planes {seed}")


@pytest.mark.parametrize("seed", range(8))
def test_few_input_planes_fused_epilogue(seed):
    """The block epilogue (scale, shift, residual, ReLU, each on or off) on
    layers of 1-4 input planes and at least 2048 sites, where the
    low-channel kernel stores its rows through LDS, against the oracle."""
    import oracle
    from paper_1706_01307_amd import inputs
    from tests.test_ops_gpu import _dev, _feats, _odt
    from tests.test_parity_gpu import RTOL_BF16, RTOL_F32, _t, _to_np, check_features
    rng = np.random.default_rng(7500 + seed)
    D = int(rng.integers(3, 5))
    size = [int(rng.integers(1, 3))] + [int(rng.choice([72, 80] if D == 3 else [24, 31]))
                                       for _ in range(D - 1)]
    c = dense_ref.random_sites(rng, size, 0.5 if D == 3 else 0.2)
    assert len(c) >= 2048
    f, s_ = [1] + [3] * (D - 1), [1] * D
    ci, co = int(rng.integers(1, 5)), int(rng.choice([16, 32, 48]))
    dtype = "bf16" if seed % 2 else "f32"
    out_dtype = "f32" if seed % 4 < 2 else "bf16"
    use_s, use_b, use_r, relu = (bool(v) for v in rng.integers(0, 2, size=4))
    if seed == 0:
        use_s = use_b = use_r = relu = True
    rb = spc.build_rulebook(spc.VSC, _t(c), size, f, s_)
    ref = oracle.Rulebook(oracle.VSC, c, size, f, s_)
    K = ref.K
    x = _feats(len(c), ci, dtype, 13 * seed + 1)
    wf = inputs.normal_f32((K, ci, co), std=1.0 / np.sqrt(K * ci), seed=13 * seed + 2)
    w = inputs.to_bf16_bits(wf) if dtype == "bf16" else wf
    scale = inputs.normal_f32((co,), std=1.0, seed=13 * seed + 3)
    shift = inputs.normal_f32((co,), std=0.5, seed=13 * seed + 4)
    res = _feats(ref.n_out, co, out_dtype, 13 * seed + 5)
    _say(f"[few planes fused {seed}] N={len(c)} C={ci}->{co} {dtype}->{out_dtype} "
         f"parts={use_s, use_b, use_r, relu}")
    odt = torch.bfloat16 if out_dtype == "bf16" else torch.float32
    y = spc.forward_fused(rb, _dev(x, dtype), _dev(w, dtype),
                          scale=_t(scale) if use_s else None, shift=_t(shift) if use_b else None,
                          residual=_dev(res, out_dtype) if use_r else None, relu=relu,
                          out_dtype=odt)
    y64, absb = ref.forward(x, w, None, in_dt=_odt(dtype))
    zo, bound = oracle.fused_epilogue(y64, absb, scale if use_s else None,
                                      shift if use_b else None, res if use_r else None,
                                      relu, _odt(out_dtype))
    rtol = RTOL_F32 if dtype == "f32" and out_dtype == "f32" else RTOL_BF16
    check_features(_to_np(y), zo, bound, rtol, "few planes fused")
