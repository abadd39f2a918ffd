"""Pins for the oracle's FGQ layer: y = s_x * sum_g alpha_g * sum_{i in g} t_i q_i.

The layer is an exact real formula, so the oracle must equal a library
convolution (torch.nn.functional.conv2d, float64, CPU) of the dequantized
activations s_x*q with the reconstructed weights alpha*t laid out in the
original [O][C][R][S] order.  That pins indexing, stride, padding, the
grouping of K and the code layout independently of the oracle's loops.
Group sums are pinned against an independent im2col built with
torch.nn.functional.unfold.
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

import fgq_inputs as fi
import oracle


def unpack_acts(q, bits, n):
    if bits == 8:
        return q[:n].astype(np.int64)
    return np.stack([q & 15, q >> 4], 1).ravel()[:n].astype(np.int64)


def reconstructed_weights(t, alpha, O, C, R, S, G):
    """alpha*t from [O][R][S][C]-ordered codes back to [O][C][R][S] float64."""
    K = R * S * C
    w = t.reshape(O, K // G, G).astype(np.float64) * alpha.astype(np.float64)[:, :, None]
    return w.reshape(O, R, S, C).transpose(0, 3, 1, 2)


def library_conv(qv, sx, B, H, W, C, w, stride, pad):
    x = torch.from_numpy(qv.reshape(B, H, W, C).transpose(0, 3, 1, 2).astype(np.float64) * float(sx))
    y = F.conv2d(x, torch.from_numpy(np.ascontiguousarray(w)), stride=stride, padding=pad)
    return y.permute(0, 2, 3, 1).reshape(-1, w.shape[0]).numpy()


CASES = [
    # B, H, W, C, O, R, S, stride, pad, G, bits
    (2, 9, 7, 16, 12, 3, 3, 1, 1, 4, 8),
    (2, 9, 7, 16, 12, 3, 3, 2, 1, 4, 8),
    (1, 11, 11, 8, 5, 1, 1, 2, 0, 8, 8),
    (2, 13, 13, 4, 6, 7, 7, 2, 3, 4, 8),     # conv1-like, C padded 3->4
    (2, 6, 5, 64, 9, 3, 3, 1, 1, 64, 8),
    (2, 6, 5, 64, 9, 3, 3, 1, 1, 64, 4),
    (3, 5, 6, 12, 7, 3, 1, 1, 0, 2, 4),
    (1, 4, 4, 6, 3, 2, 2, 1, 1, 1, 8),       # G=1 and an even kernel
]


@pytest.mark.parametrize("case", CASES)
def test_conv_equals_library_convolution(case):
    B, H, W, C, O, R, S, st, pd, G, bits = case
    w = fi.he_weights(O, C, R, S, "lib", case)
    x = fi.relu_gauss((B, H, W, C), "lib", case)
    t, alpha, _ = oracle.ternarize(w, G)
    codes = oracle.pack_codes(t)
    q, sx = oracle.quantize_act(x, bits)
    y = oracle.conv2d(q, bits, sx, (B, H, W, C), codes, alpha, O, R, S, (st, st), (pd, pd), G)
    ref = library_conv(unpack_acts(q, bits, x.size), sx, B, H, W, C,
                       reconstructed_weights(t, alpha, O, C, R, S, G), st, pd)
    assert y.shape == ref.shape
    scale = np.abs(ref).max() + 1e-30
    np.testing.assert_allclose(y, ref, rtol=2e-7, atol=1e-12 * scale)


def test_group_size_one_is_the_original_convolution():
    """G=1 has zero ternary error, so the layer equals the convolution with
    the original fp32 weights."""
    B, H, W, C, O, R, S = 2, 8, 8, 6, 5, 3, 3
    w = fi.he_weights(O, C, R, S, "g1")
    x = fi.relu_gauss((B, H, W, C), "g1")
    t, alpha, _ = oracle.ternarize(w, 1)
    q, sx = oracle.quantize_act(x, 8)
    y = oracle.conv2d(q, 8, sx, (B, H, W, C), oracle.pack_codes(t), alpha, O, R, S, (1, 1), (1, 1), 1)
    ref = library_conv(unpack_acts(q, 8, x.size), sx, B, H, W, C, w.astype(np.float64), 1, 1)
    np.testing.assert_allclose(y, ref, rtol=2e-7, atol=1e-12)


@pytest.mark.parametrize("bits", [8, 4])
def test_gemm_equals_matmul(bits):
    M, K, O, G = 37, 256, 19, 4
    w = fi.gauss_weights(O, K, 0.05, "gemm")
    x = fi.relu_gauss((M, K), "gemm")
    t, alpha, _ = oracle.ternarize(w, G)
    q, sx = oracle.quantize_act(x, bits)
    y = oracle.gemm(q, bits, sx, M, K, oracle.pack_codes(t), alpha, O, G)
    wr = t.reshape(O, K // G, G) * alpha.astype(np.float64)[:, :, None]
    ref = (unpack_acts(q, bits, x.size).reshape(M, K).astype(np.float64) * float(sx)) @ wr.reshape(O, K).T
    np.testing.assert_allclose(y, ref, rtol=2e-7, atol=1e-12 * np.abs(ref).max())


def test_group_sums_against_unfold():
    B, H, W, C, O, R, S, st, pd, G, bits = 2, 7, 6, 8, 5, 3, 3, 2, 1, 4, 8
    w = fi.he_weights(O, C, R, S, "gs")
    x = fi.relu_gauss((B, H, W, C), "gs")
    t, alpha, _ = oracle.ternarize(w, G)
    q, sx = oracle.quantize_act(x, bits)
    P = oracle.group_sums_conv(q, bits, (B, H, W, C), oracle.pack_codes(t), O, R, S, (st, st), (pd, pd), G)
    qv = torch.from_numpy(unpack_acts(q, bits, x.size).reshape(B, H, W, C).transpose(0, 3, 1, 2).astype(np.float64))
    cols = F.unfold(qv, (R, S), padding=pd, stride=st)          # [B, C*R*S (c-major), L]
    L = cols.shape[-1]
    cols = cols.reshape(B, C, R, S, L).permute(0, 4, 2, 3, 1).reshape(B * L, R * S * C).numpy()
    prod = cols[:, None, :] * t[None, :, :].astype(np.float64)    # [M][O][K]
    ref = prod.reshape(B * L, O, -1, G).sum(-1)
    np.testing.assert_array_equal(P, ref.astype(np.int64))
    assert np.abs(P).max() <= G * 255
    # a row subset is the same slice
    P2 = oracle.group_sums_conv(q, bits, (B, H, W, C), oracle.pack_codes(t), O, R, S, (st, st), (pd, pd), G,
                                row0=5, nrows=7)
    np.testing.assert_array_equal(P2, P[5:12])


@pytest.mark.parametrize("case", [(2, 9, 7, 16, 12, 3, 3, 2, 1, 4, 8), (3, 6, 6, 64, 5, 1, 1, 1, 0, 64, 4)])
def test_rows_variant_and_summand_magnitude(case):
    """conv2d_rows (a list of rows, any order, repeats allowed) gives the
    full convolution's values bit for bit, and its magnitude is
    s_x * sum_g alpha_g |P_g| from the group sums (pinned against unfold
    below), summed independently with numpy."""
    B, H, W, C, O, R, S, st, pd, G, bits = case
    w = fi.he_weights(O, C, R, S, "rows", case)
    x = fi.relu_gauss((B, H, W, C), "rows", case)
    t, a, _ = oracle.ternarize(w, G)
    codes = oracle.pack_codes(t)
    q, s = oracle.quantize_act(x, bits)
    y = oracle.conv2d(q, bits, s, x.shape, codes, a, O, R, S, (st, st), (pd, pd), G)
    M = y.shape[0]
    rows = np.random.default_rng(7).integers(0, M, 40)
    rows[:3] = [M - 1, 0, M - 1]
    yr, mag = oracle.conv2d_rows(q, bits, s, x.shape, codes, a, O, R, S, (st, st), (pd, pd), G, rows)
    np.testing.assert_array_equal(yr.view(np.uint32), y[rows].view(np.uint32))
    P = oracle.group_sums_conv(q, bits, x.shape, codes, O, R, S, (st, st), (pd, pd), G).astype(np.float64)
    ref = float(s) * np.einsum("mog,og->mo", np.abs(P[rows]), a.astype(np.float64))
    np.testing.assert_allclose(mag, ref, rtol=1e-12, atol=0)
    assert np.all(mag >= np.abs(yr.astype(np.float64)) * (1 - 1e-6))


def test_one_hot_and_all_ones_activations():
    M, K, O, G = 4, 64, 3, 4
    w = fi.gauss_weights(O, K, 1.0, "onehot")
    t, alpha, _ = oracle.ternarize(w, G)
    codes = oracle.pack_codes(t)
    # one-hot activation selects alpha*t of one weight
    for k in (0, 5, 63):
        q = np.zeros(M * K, np.uint8)
        q[2 * K + k] = 1
        y = oracle.gemm(q, 8, 1.0, M, K, codes, alpha, O, G)
        np.testing.assert_array_equal(y[2], alpha[:, k // G] * t[:, k])
        assert not y[[0, 1, 3]].any()
    # all-ones activations: P_g = T_g = sum of the group's codes
    P = oracle.group_sums_conv(np.ones(K, np.uint8), 8, (1, 1, 1, K), codes, O, 1, 1, (1, 1), (0, 0), G)
    np.testing.assert_array_equal(P[0], t.reshape(O, K // G, G).sum(-1))


def test_shape_errors():
    q = np.zeros(64, np.uint8)
    codes = np.zeros((2, 16), np.uint8)
    alpha = np.zeros((2, 16), np.float32)
    with pytest.raises(oracle.OracleError) as e:
        oracle.gemm(q, 8, 1.0, 1, 64, codes, alpha, 2, 3)   # K % G != 0
    assert e.value.code == 3
    with pytest.raises(oracle.OracleError) as e:
        oracle.gemm(q, 5, 1.0, 1, 64, codes, alpha, 2, 4)
    assert e.value.code == 4
