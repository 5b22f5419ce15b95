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
