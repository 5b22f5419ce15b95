"""Property-based pins of the oracle: random small grids, filters, strides,
densities and channel counts (hypothesis), each checked against the dense
brute-force convolution and the dense row-grid rule book of tests/dense_ref.py.
CPU only."""
import numpy as np
import pytest

hypothesis = pytest.importorskip("hypothesis")
from hypothesis import given, settings, strategies as st  # noqa: E402

import oracle  # noqa: E402
from tests import dense_ref  # noqa: E402


@st.composite
def layer_case(draw, kind):
    d = draw(st.integers(1, 3))
    ext = {1: 9, 2: 7, 3: 5}[d]
    size_sp = [draw(st.integers(1, ext)) for _ in range(d)]
    batch = draw(st.integers(1, 2))
    if kind == "vsc":
        f_sp = [draw(st.sampled_from([1, 3, 5])) for _ in range(d)]
        s_sp = [1] * d
    else:
        f_sp = [draw(st.integers(1, 3)) for _ in range(d)]
        s_sp = [draw(st.integers(1, 3)) for _ in range(d)]
    density = draw(st.floats(0.0, 1.0))
    c_in, c_out = draw(st.integers(1, 3)), draw(st.integers(1, 3))
    seed = draw(st.integers(0, 2**31 - 1))
    return d, [batch] + size_sp, [1] + f_sp, [1] + s_sp, density, c_in, c_out, seed


def _inputs(size, f, density, c_in, c_out, seed):
    rng = np.random.default_rng(seed)
    coords = dense_ref.random_sites(rng, size, density)
    K = int(np.prod(f))
    x = rng.standard_normal((len(coords), c_in)).astype(np.float32)
    w = rng.standard_normal((K, c_in, c_out)).astype(np.float32)
    b = rng.standard_normal(c_out).astype(np.float32)
    return coords, x, w, b


@settings(max_examples=80, deadline=None)
@given(layer_case("vsc"))
def test_vsc_random_cases_match_bruteforce(case):
    d, size, f, s, density, c_in, c_out, seed = case
    coords, x, w, b = _inputs(size, f, density, c_in, c_out, seed)
    rb = oracle.Rulebook(oracle.VSC, coords, size, f)
    y, absb = rb.forward(x, w, b)
    ref = dense_ref.vsc_dense(coords, size, f, x, w, b)
    np.testing.assert_allclose(y, ref, rtol=0, atol=1e-12 * (1 + np.abs(absb).max(initial=0.0)))
    R = dense_ref.rulebook_dense("vsc", coords, size, f, None, coords)
    for i in range(rb.K):
        np.testing.assert_array_equal(rb.offset_pairs(i), R[i])
    k = np.diff(rb.pair_off)
    assert np.array_equal(k, k[::-1])                       # k_i = k_{K-1-i}
    if len(coords):
        assert k[rb.K // 2] == len(coords)                  # the centre offset


@settings(max_examples=80, deadline=None)
@given(layer_case("sc"))
def test_sc_random_cases_match_bruteforce(case):
    d, size, f, s, density, c_in, c_out, seed = case
    coords, x, w, b = _inputs(size, f, density, c_in, c_out, seed)
    rb = oracle.Rulebook(oracle.SC, coords, size, f, s)
    oc, ref = dense_ref.sc_dense(coords, size, f, s, x, w, b)
    np.testing.assert_array_equal(rb.out_coords.reshape(-1, len(size)), oc.reshape(-1, len(size)))
    np.testing.assert_array_equal(rb.out_size, dense_ref.sc_extent(size, f, s))
    y, absb = rb.forward(x, w, b)
    np.testing.assert_allclose(y, ref.reshape(y.shape), rtol=0,
                               atol=1e-12 * (1 + np.abs(absb).max(initial=0.0)))
    R = dense_ref.rulebook_dense("sc", coords, size, f, s, rb.out_coords)
    for i in range(rb.K):
        np.testing.assert_array_equal(rb.offset_pairs(i), R[i])
