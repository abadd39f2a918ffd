"""GPU parity of the layer with fixed-point group scales (Sec. 4: scaling
factors quantized to an 8/4-bit fixed point; 32-bit accumulation), through
the C ABI, against the oracle.

Bar: bit-exact everywhere.  The codes A and the fractional length fl are
integers; the layer's output is defined as fp32(double(S) * (double(s_x) *
2^-fl)) of an exact integer S, which the one-plane matrix-core kernel and
the direct fallback both evaluate exactly that way; fused 8/4-bit outputs
are then the oracle's quantization of the same fp32 values.
"""
import numpy as np
import pytest
import torch

import fgq_inputs as fi
import oracle

fgq = pytest.importorskip("paper_1705_01462_amd")

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


@pytest.mark.parametrize("bits", [8, 4])
@pytest.mark.parametrize("G,shape", [(4, (64, 128, 3, 3)), (64, (96, 256, 1, 1)), (2, (8, 6, 3, 3)),
                                     (4, (1000, 2048, 1, 1))])
def test_dfp_alpha_bit_exact(bits, G, shape):
    O, C, R, S = shape
    w = fi.he_weights(O, C, R, S, "gpu-dfp", G)
    _, alpha, _ = oracle.ternarize(w, G)
    A_ref, fl_ref = oracle.dfp_alpha(alpha, bits)
    A, fl = fgq.fgq_dfp_alpha(dev(alpha), bits)
    assert int(host(fl)[0]) == fl_ref
    np.testing.assert_array_equal(host(A), A_ref)


def test_dfp_alpha_rejects_bad_scales():
    for bad in (np.nan, np.inf, -0.5):
        a = np.full(100, 0.25, np.float32)
        a[37] = bad
        with pytest.raises(fgq.FgqError) as e:
            fgq.fgq_dfp_alpha(dev(a), 8)
        assert e.value.code == 5
    A, fl = fgq.fgq_dfp_alpha(dev(np.zeros(10, np.float32)), 4)
    assert int(host(fl)[0]) == 0 and not host(A).any()


def dfp_layer(B, H, W, C, O, R, S, st, pd, G, bits, ab, tag, x=None, w=None):
    if w is None:
        w = fi.he_weights(O, C, R, S, "gpu-dfp-layer", tag)
    if x is None:
        x = fi.relu_gauss((B, H, W, C), "gpu-dfp-layer", tag)
    codes, alpha, _ = fgq.fgq_ternarize(dev(w), G)
    q, sx = fgq.fgq_quantize_act(dev(x), bits)
    K = R * S * C
    prep = fgq.fgq_prepare_weights_dfp(codes, alpha, O, K, G, ab)
    t, a, _ = oracle.ternarize(w, G)
    ref = dict(codes=oracle.pack_codes(t), alpha=a)
    ref["q"], ref["s"] = oracle.quantize_act(x, bits)
    ref["A"], ref["fl"] = oracle.dfp_alpha(a, ab)
    return codes, q, sx, prep, ref, x.shape


LAYER_CASES = [
    # B, H, W, C, O, R, S, stride, pad, G, bits, alpha_bits    (path)
    (2, 9, 7, 16, 24, 3, 3, 1, 1, 4, 8, 8),        # matrix core, ragged M and O
    (2, 9, 7, 16, 24, 3, 3, 2, 1, 4, 4, 8),        # uint4 activations, stride 2
    (3, 8, 8, 64, 100, 3, 3, 1, 1, 64, 8, 4),      # G = 64, 4-bit scales
    (2, 12, 12, 32, 64, 1, 1, 2, 0, 8, 8, 8),      # 1x1 stride 2
    (2, 15, 15, 4, 16, 7, 7, 2, 3, 4, 8, 8),       # tiny C = 4 (padded first layer)
    (2, 11, 11, 8, 33, 5, 5, 1, 2, 4, 4, 8),       # tiny C = 8, odd O
    (2, 10, 9, 128, 40, 3, 3, 1, 1, 4, 8, 8),      # C >= 128
    (2, 6, 6, 12, 10, 3, 3, 1, 1, 4, 8, 8),        # direct fallback (C % 16 != 0)
    (2, 6, 6, 6, 6, 3, 3, 1, 1, 3, 8, 4),          # direct fallback (C % 4 != 0)
]


@pytest.mark.parametrize("case", LAYER_CASES)
def test_conv2d_dfp_bit_exact(case):
    B, H, W, C, O, R, S, st, pd, G, bits, ab = case
    codes, q, sx, prep, ref, shape = dfp_layer(*case, tag=case)
    y = host(fgq.fgq_conv2d_dfp(q, bits, sx, shape, codes, prep, O, R, S, st, pd, G)).reshape(-1, O)
    y_ref = oracle.conv2d_dfp(ref["q"], bits, ref["s"], shape, ref["codes"], ref["A"], ref["fl"], O, R, S,
                              (st, st), (pd, pd), G)
    np.testing.assert_array_equal(y.view(np.uint32), y_ref.view(np.uint32))


@pytest.mark.parametrize("out_bits", [8, 4])
@pytest.mark.parametrize("case", [LAYER_CASES[0], LAYER_CASES[2], LAYER_CASES[4], LAYER_CASES[7]])
def test_conv2d_dfp_fused_bit_exact(case, out_bits):
    B, H, W, C, O, R, S, st, pd, G, bits, ab = case
    if out_bits == 4 and O % 2:
        pytest.skip("4-bit output needs even O")
    codes, q, sx, prep, ref, shape = dfp_layer(*case, tag=case)
    y_ref = oracle.conv2d_dfp(ref["q"], bits, ref["s"], shape, ref["codes"], ref["A"], ref["fl"], O, R, S,
                              (st, st), (pd, pd), G)
    s_out = np.float32(0.8 * float(y_ref.max()) / (2 ** out_bits - 1))
    sc = dev(np.array([s_out], np.float32))
    got = host(fgq.fgq_conv2d_dfp(q, bits, sx, shape, codes, prep, O, R, S, st, pd, G, out_bits, sc)).ravel()
    want = oracle.quantize_act(y_ref.ravel(), out_bits, s_out)[0]
    np.testing.assert_array_equal(got, want)


@pytest.mark.parametrize("M,K,O,G,bits,ab", [(64, 256, 128, 4, 8, 8), (77, 640, 40, 64, 8, 4),
                                             (5, 96, 7, 4, 4, 8), (300, 1280, 96, 8, 8, 8)])
def test_gemm_dfp_bit_exact(M, K, O, G, bits, ab):
    w = fi.gauss_weights(O, K, 0.05, "gpu-dfp-gemm", M, K)
    x = fi.relu_gauss((M, K), "gpu-dfp-gemm", M, K)
    codes, alpha, _ = fgq.fgq_ternarize(dev(w), G)
    q, sx = fgq.fgq_quantize_act(dev(x), bits)
    prep = fgq.fgq_prepare_weights_dfp(codes, alpha, O, K, G, ab)
    y = host(fgq.fgq_gemm_dfp(q, bits, sx, M, K, codes, prep, O, G))
    t, a, _ = oracle.ternarize(w, G)
    qr, sr = oracle.quantize_act(x, bits)
    A, fl = oracle.dfp_alpha(a, ab)
    y_ref = oracle.gemm_dfp(qr, bits, sr, M, K, oracle.pack_codes(t), A, fl, O, G)
    np.testing.assert_array_equal(y.view(np.uint32), y_ref.view(np.uint32))


def test_gemm_dfp_beyond_matrix_core_k_limit():
    """K > 65536 takes the direct path; still bit-exact."""
    M, K, O, G = 3, 65600, 5, 4
    w = fi.gauss_weights(O, K, 0.05, "gpu-dfp-bigk")
    x = fi.relu_gauss((M, K), "gpu-dfp-bigk")
    codes, alpha, _ = fgq.fgq_ternarize(dev(w), G)
    q, sx = fgq.fgq_quantize_act(dev(x), 8)
    prep = fgq.fgq_prepare_weights_dfp(codes, alpha, O, K, G, 8)
    y = host(fgq.fgq_gemm_dfp(q, 8, sx, M, K, codes, prep, O, G))
    t, a, _ = oracle.ternarize(w, G)
    qr, sr = oracle.quantize_act(x, 8)
    A, fl = oracle.dfp_alpha(a, 8)
    y_ref = oracle.gemm_dfp(qr, 8, sr, M, K, oracle.pack_codes(t), A, fl, O, G)
    np.testing.assert_array_equal(y.view(np.uint32), y_ref.view(np.uint32))


def test_dfp_all_zero_weights():
    B, H, W, C, O, R, S, G = 2, 6, 6, 16, 32, 3, 3, 4
    w = np.zeros((O, C, R, S), np.float32)
    codes, q, sx, prep, ref, shape = dfp_layer(B, H, W, C, O, R, S, 1, 1, G, 8, 8, "zeros", w=w)
    y = host(fgq.fgq_conv2d_dfp(q, 8, sx, shape, codes, prep, O, R, S, 1, 1, G))
    assert ref["fl"] == 0 and not ref["A"].any()
    assert not y.view(np.uint32).any()


@pytest.mark.parametrize("G", [4, 64])
def test_benchmark_layer_dfp_sampled_rows(G):
    """The batch-32 ResNet-50 conv3_x layer at full size; three sampled row
    ranges (all channels) against the oracle, bit-exact."""
    B, H, W, C, O, R, S = 32, 28, 28, 128, 128, 3, 3
    case = (B, H, W, C, O, R, S, 1, 1, G, 8, 8)
    codes, q, sx, prep, ref, shape = dfp_layer(*case, tag=("bench", G))
    y = host(fgq.fgq_conv2d_dfp(q, 8, sx, shape, codes, prep, O, R, S, 1, 1, G)).reshape(-1, O)
    M = y.shape[0]
    for row0 in (0, M // 2 - 64, M - 128):
        y_ref = oracle.conv2d_dfp(ref["q"], 8, ref["s"], shape, ref["codes"], ref["A"], ref["fl"], O, R, S,
                                  (1, 1), (1, 1), G, rows=(row0, 128))[row0:row0 + 128]
        np.testing.assert_array_equal(y[row0:row0 + 128].view(np.uint32), y_ref.view(np.uint32))


# ---------------------------------------------------------------------------
# First layer at 8-bit weights (Sec. 4: 8w-8a)
# ---------------------------------------------------------------------------

W8_CASES = [
    # B, H, W, C, O, R, S, stride, pad, bits
    (2, 23, 23, 4, 64, 7, 7, 2, 3, 8),      # ResNet conv1 shape, image padded to 4 channels
    (2, 9, 7, 16, 24, 3, 3, 1, 1, 8),
    (2, 11, 11, 8, 33, 5, 5, 1, 2, 4),      # tiny C = 8, uint4 input, odd O
    (1, 10, 10, 64, 96, 1, 1, 2, 0, 8),
]


@pytest.mark.parametrize("case", W8_CASES)
def test_conv2d_w8_bit_exact(case):
    B, H, W, C, O, R, S, st, pd, bits = case
    w = fi.he_weights(O, C, R, S, "gpu-w8", case)
    x = fi.relu_gauss((B, H, W, C), "gpu-w8", case)
    prep = fgq.fgq_prepare_weights_w8(dev(w))
    q, sx = fgq.fgq_quantize_act(dev(x), bits)
    y = host(fgq.fgq_conv2d_w8(q, bits, sx, x.shape, prep, O, R, S, st, pd)).reshape(-1, O)
    W8, fl = oracle.w8_quantize(w)
    qr, sr = oracle.quantize_act(x, bits)
    y_ref = oracle.conv2d_w8(qr, bits, sr, x.shape, W8, fl, O, R, S, (st, st), (pd, pd))
    np.testing.assert_array_equal(y.view(np.uint32), y_ref.view(np.uint32))
    if O % 2 == 0:
        s_out = np.float32(0.7 * float(y_ref.max()) / 255)
        got = host(fgq.fgq_conv2d_w8(q, bits, sx, x.shape, prep, O, R, S, st, pd, 8,
                                     dev(np.array([s_out], np.float32)))).ravel()
        np.testing.assert_array_equal(got, oracle.quantize_act(y_ref.ravel(), 8, s_out)[0])


def test_conv2d_w8_unsupported_and_bad_weights():
    w = fi.he_weights(8, 3, 3, 3, "gpu-w8-c3")
    prep = fgq.fgq_prepare_weights_w8(dev(w))
    q, sx = fgq.fgq_quantize_act(dev(fi.relu_gauss((1, 6, 6, 3), "gpu-w8-c3")), 8)
    with pytest.raises(fgq.FgqError) as e:
        fgq.fgq_conv2d_w8(q, 8, sx, (1, 6, 6, 3), prep, 8, 3, 3, 1, 1)
    assert e.value.code == 7
    w[3, 1, 2, 0] = np.nan
    with pytest.raises(fgq.FgqError) as e:
        fgq.fgq_prepare_weights_w8(dev(w))
    assert e.value.code == 5


@pytest.mark.parametrize("out_bits", [0, 8, 4])
@pytest.mark.parametrize("case", [LAYER_CASES[0], LAYER_CASES[2], LAYER_CASES[4], LAYER_CASES[5],
                                  LAYER_CASES[7]])
def test_conv2d_dfp_residual_bit_exact(case, out_bits):
    """The shortcut addition and ReLU in the epilogue (and the output's codes
    from it): the oracle's layer plus an fp32 addition and a ReLU, and the
    oracle's quantization of that, bit for bit."""
    B, H, W, C, O, R, S, st, pd, G, bits, ab = case
    if out_bits == 4 and O % 2:
        pytest.skip("4-bit output needs even O")
    codes, q, sx, prep, ref, shape = dfp_layer(*case, tag=case)
    y_ref = oracle.conv2d_dfp(ref["q"], bits, ref["s"], shape, ref["codes"], ref["A"], ref["fl"], O, R, S,
                              (st, st), (pd, pd), G).reshape(-1, O)
    res = fi.rng("gpu-dfp-residual", case).standard_normal(y_ref.shape).astype(np.float32)
    s = (y_ref + res).astype(np.float32)
    want = np.where(s < 0, np.float32(0), s)
    Ho, Wo = fgq.conv_out_hw(H, W, R, S, (st, st), (pd, pd))
    rd = dev(res.reshape(B, Ho, Wo, O))
    s_out = np.float32(0.8 * float(want.max()) / (2 ** out_bits - 1)) if out_bits else None
    sc = dev(np.array([s_out], np.float32)) if out_bits else None
    got = fgq.fgq_conv2d_dfp_residual(q, bits, sx, shape, codes, prep, O, R, S, st, pd, G, rd, out_bits, sc)
    y = got[0] if out_bits else got
    np.testing.assert_array_equal(host(y).reshape(-1, O).view(np.uint32), want.view(np.uint32))
    if out_bits:
        np.testing.assert_array_equal(host(got[1]).ravel(), oracle.quantize_act(want.ravel(), out_bits, s_out)[0])
