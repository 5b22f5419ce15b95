"""Seeded random layers for the rows after the hot path, against the oracle:
max / average pooling and DC on SC books, and the input and weight
gradients of VSC, SC and DC, over random extents, filters, strides,
densities, channel counts and dtypes."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

import oracle  # noqa: E402
import paper_1706_01307_amd as spc  # noqa: E402
from paper_1706_01307_amd import inputs  # noqa: E402
from tests import dense_ref  # noqa: E402
from tests.test_ops_gpu import OP, RTOL_GRAD, _dev, _feats, _odt  # noqa: E402
from tests.test_parity_gpu import (RTOL_BF16, RTOL_F32, _say, _t, _to_np,  # noqa: E402
                                   check_features)

pytestmark = pytest.mark.gpu

CHANNELS = [(1, 16), (16, 16), (32, 32), (32, 64), (64, 64), (64, 32), (5, 3), (96, 32)]


def _case(seed):
    rng = np.random.default_rng(5000 + seed)
    D = int(rng.integers(2, 5))
    op = str(rng.choice(["vsc", "sc", "dc"]))
    size = [int(rng.integers(1, 4))] + [int(rng.choice([2, 3, 5, 8, 13, 16, 31]))
                                       for _ in range(D - 1)]
    if op == "vsc":
        f = [1] + [int(rng.choice([1, 3, 3, 5])) for _ in range(D - 1)]
        s = [1] * D
    else:
        f = [1] + [int(rng.integers(1, 4)) for _ in range(D - 1)]
        s = [1] + [int(rng.integers(1, 4)) for _ in range(D - 1)]
        f = [min(fj, sz) for fj, sz in zip(f, size)]
    density = float(rng.choice([0.05, 0.2, 0.5, 1.0]))
    ci, co = CHANNELS[int(rng.integers(0, len(CHANNELS)))]
    dtype = "bf16" if (ci % 8 == 0 and co % 8 == 0 and rng.random() < 0.5) else "f32"
    c = dense_ref.random_sites(rng, size, density)
    if len(c) == 0:
        c = np.array([[int(rng.integers(0, e)) for e in size]], np.int32)
    while len(c) > 1 and len(c) * int(np.prod(f)) * ci * co > 2e8:
        c = c[::2]
    return op, c, size, f, s, ci, co, dtype


@pytest.mark.parametrize("seed", range(64))
def test_random_gradients_pooling_dc(seed):
    op, c, size, f, s, ci, co, dtype = _case(seed)
    kind = spc.VSC if op == "vsc" else spc.SC
    rtol = RTOL_F32 if dtype == "f32" else RTOL_BF16
    rb = spc.build_rulebook(kind, _t(c), size, f, s, transpose=(op != "vsc"))
    ref = oracle.Rulebook(kind, c, size, f, s)
    K = ref.K
    _say(f"[random ops {seed}] {op} N={len(c)} -> {ref.n_out} size={size} f={f} s={s} "
         f"C={ci}->{co} {dtype}")
    in_rows = ref.n_out if op == "dc" else ref.n_in
    out_rows = ref.n_in if op == "dc" else ref.n_out
    x = _feats(in_rows, ci, dtype, 7 * seed + 1)
    dy = _feats(out_rows, co, dtype, 7 * seed + 2)
    wf = inputs.normal_f32((K, ci, co), std=1.0 / np.sqrt(K * ci), seed=7 * seed + 3)
    w = inputs.to_bf16_bits(wf) if dtype == "bf16" else wf
    if op == "dc":
        b = inputs.normal_f32((co,), std=0.1, seed=7 * seed + 4)
        y = spc.dc_forward(rb, _dev(x, dtype), _dev(w, dtype), _t(b))
        yo, absb = ref.dc_forward(x, w, b, in_dt=_odt(dtype))
        check_features(_to_np(y), yo, absb, rtol, "DC")
    if op == "sc":
        xp = _feats(ref.n_in, ci, dtype, 7 * seed + 5)
        mp = spc.pool_forward(rb, _dev(xp, dtype), spc.POOL_MAX)
        ap = spc.pool_forward(rb, _dev(xp, dtype), spc.POOL_AVG)
        mo, _ = ref.pool(xp, oracle.POOL_MAX, _odt(dtype))
        ao, aab = ref.pool(xp, oracle.POOL_AVG, _odt(dtype))
        got = (mp.view(torch.int16).cpu().numpy().view(np.uint16) if dtype == "bf16"
               else mp.cpu().numpy())
        np.testing.assert_array_equal(got, oracle.round_to(mo, _odt(dtype)))
        check_features(_to_np(ap), ao, aab, rtol, "AP")
    dx = spc.backward_data(rb, OP[op][0], _dev(dy, dtype), _dev(w, dtype))
    dxo, adx = ref.backward_data(OP[op][1], dy, w, _odt(dtype))
    check_features(_to_np(dx), dxo, adx, rtol, "dx")
    dw, db = spc.backward_weight(rb, OP[op][0], _dev(x, dtype), _dev(dy, dtype), ci, co)
    dwo, dbo, aw, ab = ref.backward_weight(OP[op][1], x, dy, ci, co, _odt(dtype))
    check_features(dw.cpu().numpy(), dwo, aw, RTOL_GRAD, "dw")
    check_features(db.cpu().numpy(), dbo, ab, RTOL_GRAD, "db")
