"""Rule books built on the output sites of an SC rule book (a chain of
levels) without the host waiting.  Each chained book is compared with the
oracle's book built on the oracle's own SC output sites (bit for bit, pairs
canonicalised per R_i) and its forward with the oracle's forward; it is also
compared with the library's book built from the exported output sites, also
for the hash-table path (which reads the count on the host) and a
three-level chain."""
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")

import oracle  # noqa: E402
import paper_1706_01307_amd as spc  # noqa: E402
from paper_1706_01307_amd import inputs  # noqa: E402
from tests.rb_check import check_rulebook  # noqa: E402
from tests.test_parity_gpu import RTOL_BF16, _bf16_tensor, _t, _to_np, check_features  # noqa: E402

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _feat_bits(n, C, seed):
    return inputs.to_bf16_bits(inputs.normal_f32((n, C), seed=seed))


def _weight_bits(K, ci, co, seed):
    return inputs.to_bf16_bits(inputs.normal_f32((K, ci, co), std=1.0 / np.sqrt(K * ci),
                                                 seed=seed))


def _feats(n, C, seed):
    return _bf16_tensor(_feat_bits(n, C, seed))


def _weights(K, ci, co, seed):
    return _bf16_tensor(_weight_bits(K, ci, co, seed))


def _oracle_kind(kind):
    return oracle.VSC if kind == spc.VSC else oracle.SC


def _same_as_oracle(rb, ref):
    """A (chained) GPU book against an oracle.Rulebook."""
    assert rb.status() == spc.OK
    assert rb.n_in == ref.n_in and rb.n_out == ref.n_out
    oc, pr = rb.export()
    check_rulebook(oc.cpu().numpy(), pr.cpu().numpy(), rb.pair_off, ref)


def _same_book(rb, ref):
    assert rb.status() == spc.OK
    assert rb.n_in == ref.n_in and rb.n_out == ref.n_out
    np.testing.assert_array_equal(rb.pair_off, ref.pair_off)
    oc, pr = rb.export()
    oc_r, pr_r = ref.export()
    assert torch.equal(oc, oc_r) and torch.equal(pr, pr_r)


def _forward(rb, x, w, C_out, out_rows):
    y = torch.zeros((out_rows, C_out), dtype=torch.bfloat16, device="cuda")
    fwd = spc.vsc_forward if rb.kind == spc.VSC else spc.sc_forward
    return fwd(rb, x, w, None, out=y)


@pytest.mark.parametrize("path", ["grid", "grid3", "hash"])
@pytest.mark.parametrize("kind,f,s", [(spc.VSC, [1, 3, 3, 3], None),
                                      (spc.SC, [1, 2, 2, 2], [1, 2, 2, 2]),
                                      (spc.SC, [1, 3, 3, 3], [1, 2, 2, 2])])
def test_chained_book_equals_book_on_exported_sites(monkeypatch, path, kind, f, s):
    monkeypatch.setenv("SPCONV_RULEBOOK", path)
    c = inputs.surfaces(2, 48, 6, 20, seed=9, variant="literal")
    size = [2, 48, 48, 48]
    parent = spc.build_rulebook(spc.SC, _t(c), size, [1, 2, 2, 2], [1, 2, 2, 2], sync=False)
    rb = spc.build_rulebook_on(parent, kind, f, s, sync=False)
    nb_in, nb_out = rb.bounds()
    K = int(np.prod(f))
    # features of the parent's outputs, allocated by the bound (no wait yet)
    x = _feats(nb_in, 32, 31)
    w = _weights(K, 32, 32, 32)
    y = _forward(rb, x, w, 32, nb_out)
    _say(f"[chain] {path} kind={kind} f={f} parent n_out={parent.n_out} bounds={nb_in},{nb_out}")
    # the oracle's chain: its own SC output sites feed its next book
    o_parent = oracle.Rulebook(oracle.SC, c, size, [1, 2, 2, 2], [1, 2, 2, 2])
    o_book = oracle.Rulebook(_oracle_kind(kind), o_parent.out_coords, o_parent.out_size, f, s)
    _same_as_oracle(rb, o_book)
    yo, absb = o_book.forward(_feat_bits(nb_in, 32, 31)[:o_book.n_in],
                              _weight_bits(K, 32, 32, 32), None, in_dt=oracle.BF16)
    check_features(_to_np(y[:o_book.n_out]), yo, absb, RTOL_BF16, "chained forward")
    # and the library's own book built from the exported sites
    oc, _ = parent.export()
    ref = spc.build_rulebook(kind, oc, parent.out_spatial_size, f, s)
    assert nb_in >= parent.n_out and nb_out >= ref.n_out
    _same_book(rb, ref)
    y_ref = _forward(ref, x[:parent.n_out].contiguous(), w, 32, ref.n_out)
    assert torch.equal(y[:ref.n_out], y_ref)


def test_three_level_chain_without_waiting():
    c = inputs.surfaces(2, 64, 8, 28, seed=10, variant="literal")
    size = [2, 64, 64, 64]
    f2 = [1, 2, 2, 2]
    levels = [spc.build_rulebook(spc.SC, _t(c), size, f2, f2, sync=False)]
    vsc = []
    for _ in range(2):
        vsc.append(spc.build_rulebook_on(levels[-1], spc.VSC, [1, 3, 3, 3], sync=False))
        levels.append(spc.build_rulebook_on(levels[-1], spc.SC, f2, f2, sync=False))
    # every level against the oracle's chain on its own output sites
    o_sites, o_size = c, size
    for lvl in range(3):
        o_sc = oracle.Rulebook(oracle.SC, o_sites, o_size, f2, f2)
        _same_as_oracle(levels[lvl], o_sc)
        o_sites, o_size = o_sc.out_coords, o_sc.out_size
        if lvl < 2:
            _same_as_oracle(vsc[lvl], oracle.Rulebook(oracle.VSC, o_sites, o_size, [1, 3, 3, 3]))
    # and with the library's books built from exported sites
    sites, sz = _t(c), size
    ref_sc = spc.build_rulebook(spc.SC, sites, sz, f2, f2)
    for lvl in range(3):
        _same_book(levels[lvl], ref_sc)
        sites, _ = ref_sc.export()
        sz = ref_sc.out_spatial_size
        if lvl < 2:
            _same_book(vsc[lvl], spc.build_rulebook(spc.VSC, sites, sz, [1, 3, 3, 3]))
            ref_sc = spc.build_rulebook(spc.SC, sites, sz, f2, f2)


def test_chained_build_argument_errors():
    c = inputs.pen_strokes(2, 64, seed=3)
    vsc = spc.build_rulebook(spc.VSC, _t(c), [2, 64, 64], [1, 3, 3])
    with pytest.raises(ValueError):
        spc.build_rulebook_on(vsc, spc.VSC, [1, 3, 3])
    sc = spc.build_rulebook(spc.SC, _t(c), [2, 64, 64], [1, 2, 2], [1, 2, 2])
    lib = spc._lib.load()
    import ctypes
    h = ctypes.c_void_p()
    f = np.asarray([1, 3, 3], np.int32)
    one = np.ones(3, np.int32)
    assert lib.spconv_build_rulebook_on(vsc.handle, 0, f.ctypes.data, one.ctypes.data, 0, None,
                                        ctypes.byref(h)) == spc.EINVAL
    assert lib.spconv_build_rulebook_on(sc.handle, 1, f.ctypes.data, one.ctypes.data,
                                        spc.BUILD_TRANSPOSE, None, ctypes.byref(h)) == spc.EINVAL
    assert h.value is None


@pytest.mark.parametrize("seed", range(24))
def test_random_chains(seed):
    """Random 4-D grids, densities and filters: a book chained on an SC
    book equals the book built from the exported sites."""
    from tests import dense_ref
    rng = np.random.default_rng(700 + seed)
    size = [int(rng.integers(1, 4))] + [int(rng.choice([2, 4, 7, 16, 33])) for _ in range(3)]
    c = dense_ref.random_sites(rng, size, float(rng.choice([0.05, 0.3, 0.9])))
    if len(c) == 0:
        c = np.zeros((1, 4), np.int32)
    fp = [1] + [int(rng.integers(1, min(3, e) + 1)) for e in size[1:]]
    sp = [1] + [int(rng.integers(1, 3)) for _ in range(3)]
    parent = spc.build_rulebook(spc.SC, _t(c), size, fp, sp, sync=False)
    if rng.random() < 0.5:
        kind, f, s = spc.VSC, [1] + [int(rng.choice([1, 3])) for _ in range(3)], None
    else:
        kind, f, s = spc.SC, [1, 2, 2, 2], [1, 2, 2, 2]
    osz = parent.out_spatial_size
    if kind == spc.SC and any(e < 2 for e in osz[1:]):
        kind, f, s = spc.VSC, [1, 3, 3, 3], None
    rb = spc.build_rulebook_on(parent, kind, f, s, sync=False)
    _say(f"[random chain {seed}] size={size} fp={fp} sp={sp} -> kind={kind} f={f}")
    o_parent = oracle.Rulebook(oracle.SC, c, size, fp, sp)
    _same_as_oracle(parent, o_parent)
    _same_as_oracle(rb, oracle.Rulebook(_oracle_kind(kind), o_parent.out_coords,
                                        o_parent.out_size, f, s or [1, 1, 1, 1]))
    oc, _ = parent.export()
    ref = spc.build_rulebook(kind, oc, osz, f, s)
    _same_book(rb, ref)
