"""The convolution with a residual block's shortcut addition and ReLU fused
into its epilogue (fgq_conv2d_residual), through the C ABI, on every kernel
family: folded (G=4, tiny C), per-group (G=64, uint8 and uint4), the
row-walking kernel (1x1, K=64, many row tiles), the direct kernel (no
prepared buffer, C % 4 != 0), staged (O % 4 == 0) and direct (O % 4 != 0)
stores.

Bars: bit-identical to fgq_conv2d followed by an fp32 addition and a ReLU
(same kernels and arithmetic); the same in place (y is the residual); with
the output's 8- or 4-bit codes written by the same epilogue
(fgq_conv2d_residual_q), the same fp32 output and codes bit-identical to
fgq_quantize_act of it at the same scale;
against the oracle's layer on sampled rows plus the same addition and ReLU,
within the layer tolerance (1e-5 of the summand magnitude) plus the
addition's rounding.
"""
import numpy as np
import pytest
import torch

import fgq_inputs as fi
import oracle

fgq = pytest.importorskip("paper_1705_01462_amd")

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

TOL = 1e-5


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def add_relu(y, r):
    s = (y + r).astype(np.float32)
    return np.where(s < 0, np.float32(0), s)


CASES = [
    # B, H, W, C, O, R, S, stride, pad, G, bits
    (2, 9, 7, 16, 24, 3, 3, 1, 1, 4, 8),
    (3, 8, 8, 64, 100, 3, 3, 1, 1, 64, 8),
    (3, 8, 8, 64, 98, 3, 3, 2, 1, 64, 4),        # O % 4 != 0: direct stores
    (2, 15, 15, 4, 16, 7, 7, 2, 3, 4, 8),        # tiny C
    (16, 56, 56, 64, 256, 1, 1, 1, 0, 4, 8),     # K = 64 over 1568 tiles: row-walking kernel
    (2, 6, 6, 6, 6, 3, 3, 1, 1, 3, 8),           # direct path only (C % 4 != 0)
    (32, 28, 28, 128, 128, 3, 3, 1, 1, 4, 8),    # benchmark layer, G=4
]


@pytest.mark.parametrize("prepared_path", [True, False], ids=["matrix-core", "direct"])
@pytest.mark.parametrize("case", CASES)
def test_residual_epilogue(case, prepared_path):
    B, H, W, C, O, R, S, st, pd, G, bits = case
    w = fi.he_weights(O, C, R, S, "residual", case)
    x = fi.relu_gauss((B, H, W, C), "residual", case)
    codes, alpha, _ = fgq.fgq_ternarize(dev(w), G)
    q, sx = fgq.fgq_quantize_act(dev(x), bits)
    K = R * S * C
    prep = fgq.fgq_prepare_weights(codes, alpha, O, K, G) if prepared_path else None
    shape = (B, H, W, C)
    Ho, Wo = fgq.conv_out_hw(H, W, R, S, (st, st), (pd, pd))
    res = fi.rng("residual-shortcut", case).standard_normal((B, Ho, Wo, O)).astype(np.float32)
    y = fgq.fgq_conv2d(q, bits, sx, shape, codes, alpha, O, R, S, st, pd, G, prepared=prep)
    rd = dev(res)
    yr = fgq.fgq_conv2d_residual(q, bits, sx, shape, codes, alpha, O, R, S, st, pd, G, rd, prepared=prep)
    got = host(yr).reshape(-1, O)
    np.testing.assert_array_equal(got, add_relu(host(y).reshape(-1, O), res.reshape(-1, O)))
    assert (got == 0).any() and (got > 0).any()
    # in place: the residual buffer receives the result
    fgq.fgq_conv2d_residual(q, bits, sx, shape, codes, alpha, O, R, S, st, pd, G, rd, prepared=prep, y=rd)
    np.testing.assert_array_equal(host(rd).reshape(-1, O), got)
    # the output's codes from the same epilogue (the next block's input)
    sc = dev(np.array([np.float32(0.8 * float(got.max()) / 255.0)], np.float32))
    for ob in (8, 4):
        if ob == 4 and O % 2:
            continue
        rd2 = dev(res)
        scb = sc if ob == 8 else dev(np.array([np.float32(0.8 * float(got.max()) / 15.0)], np.float32))
        y2, q2 = fgq.fgq_conv2d_residual_q(q, bits, sx, shape, codes, alpha, O, R, S, st, pd, G, rd2, ob, scb,
                                           prepared=prep)
        np.testing.assert_array_equal(host(y2).reshape(-1, O), got)
        qref, _ = fgq.fgq_quantize_act(y2.reshape(-1), ob, scale_in=scb)
        np.testing.assert_array_equal(host(q2).ravel(), host(qref))
    # the residual tensor must match the output's size
    with pytest.raises(ValueError):
        fgq.fgq_conv2d_residual(q, bits, sx, shape, codes, alpha, O, R, S, st, pd, G, rd.reshape(-1)[:-1],
                                prepared=prep)

    # against the oracle's layer on sampled rows
    t, a, _ = oracle.ternarize(w, G)
    q_ref, s_ref = oracle.quantize_act(x, bits)
    M = got.shape[0]
    r = fi.rng("residual-rows", case)
    rows = np.unique(np.concatenate([[0, M - 1], r.integers(0, M, min(M, 256))])).astype(np.int64)
    y_ref, mag = oracle.conv2d_rows(q_ref, bits, s_ref, x.shape, oracle.pack_codes(t), a, O, R, S, (st, st),
                                    (pd, pd), G, rows)
    want = add_relu(y_ref, res.reshape(-1, O)[rows])
    s = np.abs(y_ref.astype(np.float64) + res.reshape(-1, O)[rows])
    bound = TOL * mag + s * 2.0 ** -23
    err = np.abs(got[rows].astype(np.float64) - want)
    assert np.all(err <= bound), f"max excess {float(np.max(err - bound)):.3e}"
