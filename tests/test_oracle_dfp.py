"""Pins for the oracle's fixed-point group scales and the layer that uses them
(Sec. 4: the scaling factors quantized to an 8/4-bit fixed point; 32-bit
accumulation).

* orc_dfp_alpha: hand-worked examples (tests/golden/dfp_alpha_examples.txt),
  and on ternarized He weights the defining properties checked in exact
  rational arithmetic: A in range, every unclamped A the nearest code to
  alpha * 2^fl, and the largest alpha landing in (2^(b-2), 2^(b-1)] after
  scaling (integer length ceil(log2 amax) + 1).
* orc_conv2d_dfp / orc_gemm_dfp: equal, bit for bit, to the general oracle
  layer (itself pinned against a library convolution) run with the
  dequantized scales A * 2^-fl, and to an exact rational evaluation of
  s_x * 2^-fl * sum_k A t q on small cases.
"""
import os
from fractions import Fraction

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import fgq_inputs as fi
import oracle

HERE = os.path.dirname(os.path.abspath(__file__))


def golden_examples():
    rows = []
    for line in open(os.path.join(HERE, "golden", "dfp_alpha_examples.txt")):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        bits, alphas, fl, A = (f.strip() for f in line.split(";"))
        rows.append((int(bits), [float(v) for v in alphas.split()], int(fl), [int(v) for v in A.split()]))
    return rows


@pytest.mark.parametrize("bits,alphas,fl,A", golden_examples())
def test_dfp_alpha_worked_examples(bits, alphas, fl, A):
    got_A, got_fl = oracle.dfp_alpha(np.array(alphas, np.float32), bits)
    assert got_fl == fl
    assert got_A.tolist() == A


@pytest.mark.parametrize("bits", [8, 4])
@pytest.mark.parametrize("G", [4, 64])
def test_dfp_alpha_properties(bits, G):
    w = fi.he_weights(64, 128, 3, 3, "dfp", bits, G)
    _, alpha, _ = oracle.ternarize(w, G)
    A, fl = oracle.dfp_alpha(alpha, bits)
    top = 2 ** (bits - 1) - 1
    assert A.min() >= 0 and A.max() <= top
    scale = Fraction(2) ** fl
    amax = Fraction(float(alpha.max()))
    assert Fraction(2 ** (bits - 2)) < amax * scale <= Fraction(2 ** (bits - 1))
    for a, code in zip(alpha.ravel()[:2000], A.ravel()[:2000]):
        v = Fraction(float(a)) * scale
        if code < top:
            assert abs(v - int(code)) <= Fraction(1, 2)
        else:
            assert v >= top - Fraction(1, 2)


def test_dfp_alpha_rejects_nonfinite():
    with pytest.raises(oracle.OracleError):
        oracle.dfp_alpha(np.array([0.5, np.nan], np.float32), 8)
    with pytest.raises(oracle.OracleError):
        oracle.dfp_alpha(np.array([0.5, -0.25], np.float32), 8)


CASES = [
    # B, H, W, C, O, R, S, stride, pad, G, bits, alpha_bits
    (2, 9, 7, 16, 12, 3, 3, 1, 1, 4, 8, 8),
    (2, 9, 7, 16, 12, 3, 3, 2, 1, 4, 4, 4),
    (2, 13, 13, 4, 6, 7, 7, 2, 3, 4, 8, 8),
    (2, 6, 5, 64, 9, 3, 3, 1, 1, 64, 8, 8),
    (3, 5, 6, 12, 7, 3, 1, 1, 0, 2, 4, 8),
]


@pytest.mark.parametrize("case", CASES)
def test_conv_dfp_equals_general_layer_with_quantized_scales(case):
    B, H, W, C, O, R, S, st, pd, G, bits, ab = case
    w = fi.he_weights(O, C, R, S, "dfp-layer", case)
    x = fi.relu_gauss((B, H, W, C), "dfp-layer", case)
    t, alpha, _ = oracle.ternarize(w, G)
    codes = oracle.pack_codes(t)
    q, sx = oracle.quantize_act(x, bits)
    A, fl = oracle.dfp_alpha(alpha, ab)
    alpha_q = (A.astype(np.float64) * 2.0 ** -fl).astype(np.float32)
    assert np.array_equal(alpha_q.astype(np.float64), A.astype(np.float64) * 2.0 ** -fl)
    y_dfp = oracle.conv2d_dfp(q, bits, sx, x.shape, codes, A, fl, O, R, S, (st, st), (pd, pd), G)
    y_gen = oracle.conv2d(q, bits, sx, x.shape, codes, alpha_q, O, R, S, (st, st), (pd, pd), G)
    np.testing.assert_array_equal(y_dfp.view(np.uint32), y_gen.view(np.uint32))


def test_gemm_dfp_equals_general_layer_with_quantized_scales():
    M, K, O, G = 37, 96, 20, 4
    w = fi.gauss_weights(O, K, 0.05, "dfp-gemm")
    x = fi.relu_gauss((M, K), "dfp-gemm")
    t, alpha, _ = oracle.ternarize(w, G)
    codes = oracle.pack_codes(t)
    q, sx = oracle.quantize_act(x, 8)
    A, fl = oracle.dfp_alpha(alpha, 8)
    alpha_q = (A.astype(np.float64) * 2.0 ** -fl).astype(np.float32)
    y_dfp = oracle.gemm_dfp(q, 8, sx, M, K, codes, A, fl, O, G)
    y_gen = oracle.gemm(q, 8, sx, M, K, codes, alpha_q, O, G)
    np.testing.assert_array_equal(y_dfp.view(np.uint32), y_gen.view(np.uint32))


def test_conv_dfp_exact_rational():
    """A small layer evaluated with Python integers and Fractions; the
    integer sums come from an im2col built by torch unfold."""
    B, H, W, C, O, R, S, st, pd, G, bits = 1, 5, 4, 8, 3, 3, 3, 1, 1, 4, 8
    w = fi.he_weights(O, C, R, S, "dfp-exact")
    x = fi.relu_gauss((B, H, W, C), "dfp-exact")
    t, alpha, _ = oracle.ternarize(w, G)
    codes = oracle.pack_codes(t)
    q, sx = oracle.quantize_act(x, bits)
    A, fl = oracle.dfp_alpha(alpha, 8)
    y = oracle.conv2d_dfp(q, bits, sx, x.shape, codes, A, fl, O, R, S, (st, st), (pd, pd), G)
    K = R * S * C
    wq = (t.reshape(O, K // G, G).astype(np.int64) * A.astype(np.int64)[:, :, None]).reshape(O, R, S, C)
    xin = torch.from_numpy(q.astype(np.int64).reshape(B, H, W, C).transpose(0, 3, 1, 2).astype(np.float64))
    cols = F.unfold(xin, (R, S), padding=pd, stride=st)[0].numpy().round().astype(np.int64)  # [C*R*S][L]
    wmat = wq.transpose(0, 3, 1, 2).reshape(O, C * R * S)
    Ssum = wmat @ cols  # [O][L], exact int64
    for o in range(O):
        for m in range(Ssum.shape[1]):
            exact = Fraction(float(sx)) * int(Ssum[o, m]) / Fraction(2) ** fl
            assert abs(int(Ssum[o, m])) < 2 ** 29
            assert np.float32(float(exact)) == y[m, o]


# ---------------------------------------------------------------------------
# First layer at 8-bit weights (Sec. 4: 8w-8a)
# ---------------------------------------------------------------------------

def w8_examples():
    rows = []
    for line in open(os.path.join(HERE, "golden", "w8_weight_examples.txt")):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        ws, fl, W8 = (f.strip() for f in line.split(";"))
        rows.append(([float(v) for v in ws.split()], int(fl), [int(v) for v in W8.split()]))
    return rows


@pytest.mark.parametrize("ws,fl,W8", w8_examples())
def test_w8_worked_examples(ws, fl, W8):
    got, got_fl = oracle.w8_quantize(np.array(ws, np.float32))
    assert got_fl == fl
    assert got.tolist() == W8


def test_w8_properties():
    w = fi.he_weights(64, 4, 7, 7, "w8-props")
    W8, fl = oracle.w8_quantize(w)
    scale = Fraction(2) ** fl
    wmax = Fraction(float(np.abs(w).max()))
    assert Fraction(64) < wmax * scale <= Fraction(128)
    for a, code in zip(w.ravel(), W8.ravel()):
        v = Fraction(float(a)) * scale
        if -128 < code < 127:
            assert abs(v - int(code)) <= Fraction(1, 2)
    with pytest.raises(oracle.OracleError):
        oracle.w8_quantize(np.array([0.1, np.inf], np.float32))


@pytest.mark.parametrize("case", [(2, 15, 15, 4, 16, 7, 7, 2, 3, 8), (2, 9, 7, 16, 12, 3, 3, 1, 1, 4),
                                  (1, 8, 8, 3, 8, 3, 3, 2, 1, 8)])
def test_conv_w8_equals_integer_convolution(case):
    """S from a float64 library convolution of the integer weights and codes
    (every partial sum is an integer below 2^53, so exact), then the output
    formula evaluated with exact rationals."""
    B, H, W, C, O, R, S, st, pd, bits = case
    w = fi.he_weights(O, C, R, S, "w8-lib", case)
    x = fi.relu_gauss((B, H, W, C), "w8-lib", case)
    W8, fl = oracle.w8_quantize(w)
    q, sx = oracle.quantize_act(x, bits)
    y = oracle.conv2d_w8(q, bits, sx, x.shape, W8, fl, O, R, S, (st, st), (pd, pd))
    n = B * H * W * C
    qv = q[:n].astype(np.int64) if bits == 8 else np.stack([q & 15, q >> 4], 1).ravel()[:n].astype(np.int64)
    xin = torch.from_numpy(qv.reshape(B, H, W, C).transpose(0, 3, 1, 2).astype(np.float64))
    Sint = F.conv2d(xin, torch.from_numpy(W8.astype(np.float64)), stride=st, padding=pd)
    Sint = Sint.permute(0, 2, 3, 1).reshape(-1, O).numpy()
    assert np.all(np.abs(Sint) < 2 ** 29)
    for m in range(0, Sint.shape[0], max(1, Sint.shape[0] // 40)):
        for o in range(O):
            exact = Fraction(float(sx)) * int(round(Sint[m, o])) / Fraction(2) ** fl
            assert np.float32(float(exact)) == y[m, o]
