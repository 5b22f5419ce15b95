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
    path = str(rng.choice(["grid", "hash"]))
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
