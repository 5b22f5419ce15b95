"""GPU parity of pooling, DC, the gradients and the fused epilogue at the
sizes `bench.py --ops` times them, built the same way (SC book with its
transposed form, preallocated outputs, the same kernels).

* level 0 of the 4 x 256^3 encoder (1.70 M sites -> 0.51 M through 2^3
  stride 2): MP bit for bit and AP over every output row; DC, the SC input
  gradient and the SC weight and bias gradients over every entry.
* the 8 x 128^3 headline VSC layer (0.90 M sites, 64 -> 64): every row of
  the input gradient (a VSC forward with the flipped, transposed weights,
  an identity pinned on small cases), all 27 W^i of the weight gradient and
  the whole bias gradient, and every row of the forward with the block
  epilogue fused.
"""
import sys
import time

import numpy as np
import pytest

torch = pytest.importorskip("torch")

import oracle  # noqa: E402
import paper_1706_01307_amd as spc  # noqa: E402
from paper_1706_01307_amd import inputs  # noqa: E402
from tests.test_parity_gpu import RTOL_BF16, _bf16_tensor, _t, _to_np, check_features  # noqa: E402

pytestmark = pytest.mark.gpu
RTOL_GRAD = 1e-4


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _bits(n, c, seed, std=1.0):
    return inputs.to_bf16_bits(inputs.normal_f32((n, c), std=std, seed=seed))


def _wbits(K, ci, co, seed):
    return inputs.to_bf16_bits(inputs.normal_f32((K, ci, co), std=1.0 / np.sqrt(K * ci),
                                                 seed=seed))


def test_fullsize_encoder_level0_pool_dc_and_sc_gradients():
    t0 = time.time()
    wl = inputs.make_workload("surf256x4_unet_enc_bf16")
    n_in = len(wl.coords)
    f2 = [1, 2, 2, 2]
    rb = spc.build_rulebook(spc.SC, _t(wl.coords), wl.spatial_size, f2, f2, transpose=True)
    ref = oracle.Rulebook(oracle.SC, wl.coords, wl.spatial_size, f2, f2)
    n_out, K = ref.n_out, ref.K
    assert rb.n_out == n_out
    _say(f"[level0] {n_in} -> {n_out} sites, books built ({time.time() - t0:.1f}s)")

    x = _bits(n_in, 32, 21)
    for mode in (spc.POOL_MAX, spc.POOL_AVG):
        y = spc.pool_forward(rb, _bf16_tensor(x), mode)
        yo, absb = ref.pool(x, mode, oracle.BF16)
        if mode == spc.POOL_MAX:
            want = inputs.bf16_bits_to_f32(oracle.round_to(yo, oracle.BF16))
            np.testing.assert_array_equal(_to_np(y), want)      # MP is exact
        else:
            check_features(_to_np(y), yo, absb, RTOL_BF16, "AP")
    _say(f"[level0] pooling ok ({time.time() - t0:.1f}s)")

    ci, co = 64, 32
    xd, wd = _bits(n_out, ci, 22), _wbits(K, ci, co, 23)
    yd = spc.dc_forward(rb, _bf16_tensor(xd), _bf16_tensor(wd))
    yo, absb = ref.dc_forward(xd, wd, None, in_dt=oracle.BF16)
    check_features(_to_np(yd), yo, absb, RTOL_BF16, "DC")
    del yo, absb
    _say(f"[level0] DC ok ({time.time() - t0:.1f}s)")

    wsc, dysc = _wbits(K, co, ci, 24), _bits(n_out, ci, 25)
    dx = spc.backward_data(rb, spc.OP_SC, _bf16_tensor(dysc), _bf16_tensor(wsc))
    dxo, absb = ref.backward_data(oracle.SC, dysc, wsc, oracle.BF16)
    check_features(_to_np(dx), dxo, absb, RTOL_BF16, "SC dx")
    del dxo, absb
    _say(f"[level0] SC input gradient ok ({time.time() - t0:.1f}s)")

    xsc = _bits(n_in, co, 26)
    dw, db = spc.backward_weight(rb, spc.OP_SC, _bf16_tensor(xsc), _bf16_tensor(dysc), co, ci)
    dwo, dbo, aw, ab = ref.backward_weight(oracle.SC, xsc, dysc, co, ci, oracle.BF16)
    check_features(dw.cpu().numpy(), dwo, aw, RTOL_GRAD, "SC dw")
    check_features(db.cpu().numpy(), dbo, ab, RTOL_GRAD, "SC db")
    _say(f"[level0] SC weight gradient ok ({time.time() - t0:.1f}s)")


def test_fullsize_headline_gradients_and_fused_forward():
    t0 = time.time()
    wl = inputs.make_workload("surf128x8_vsc3_c64_bf16")
    N = len(wl.coords)
    f = [1, 3, 3, 3]
    rb = spc.build_rulebook(spc.VSC, _t(wl.coords), wl.spatial_size, f)
    ref = oracle.Rulebook(oracle.VSC, wl.coords, wl.spatial_size, f)
    K, C = 27, 64
    _say(f"[headline] N={N}, books built ({time.time() - t0:.1f}s)")

    w, dy, xv = _wbits(K, C, C, 31), _bits(N, C, 32), _bits(N, C, 33)
    dx = spc.backward_data(rb, spc.OP_VSC, _bf16_tensor(dy), _bf16_tensor(w))
    w_flip = np.ascontiguousarray(w[::-1].transpose(0, 2, 1))
    dxo, absb = ref.forward(dy, w_flip, None, in_dt=oracle.BF16)
    check_features(_to_np(dx), dxo, absb, RTOL_BF16, "VSC dx")
    del dxo, absb
    _say(f"[headline] VSC input gradient ok ({time.time() - t0:.1f}s)")

    dw, db = spc.backward_weight(rb, spc.OP_VSC, _bf16_tensor(xv), _bf16_tensor(dy), C, C)
    dwo, dbo, aw, ab = ref.backward_weight(oracle.VSC, xv, dy, C, C, oracle.BF16)
    check_features(dw.cpu().numpy(), dwo, aw, RTOL_GRAD, "VSC dw")
    check_features(db.cpu().numpy(), dbo, ab, RTOL_GRAD, "VSC db")
    _say(f"[headline] VSC weight gradient ok ({time.time() - t0:.1f}s)")

    scale = inputs.normal_f32((C,), seed=34)
    shift = inputs.normal_f32((C,), std=0.5, seed=35)
    res = _bits(N, C, 36)
    y = spc.forward_fused(rb, _bf16_tensor(xv), _bf16_tensor(w), _t(scale), _t(shift),
                          _bf16_tensor(res), True)
    yo, absb = ref.forward(xv, w, None, in_dt=oracle.BF16)
    zo, bound = oracle.fused_epilogue(yo, absb, scale, shift, res, True, oracle.BF16)
    check_features(_to_np(y), zo, bound, RTOL_BF16, "fused")
    _say(f"[headline] fused forward ok ({time.time() - t0:.1f}s)")
