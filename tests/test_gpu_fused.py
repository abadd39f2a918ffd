"""The layers with the next layer's quantization fused into the epilogue
(fgq_conv2d_q / fgq_gemm_q), through the C ABI.

Bars: bit-identical to fgq_conv2d followed by fgq_quantize_act with the same
scale (same kernels and arithmetic), on every path; against the oracle
(its layer output quantized by its own quantize_act), bit-exact on the
direct path and, on the matrix-core paths, equal except where the exact
value lies within the layer tolerance of a rounding boundary, where the
codes may differ by one.
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


def unpack(codes, out_bits, O):
    if out_bits == 8:
        return codes.reshape(-1, O).astype(np.int64)
    c = codes.reshape(-1, O // 2)
    out = np.empty((c.shape[0], O), np.int64)
    out[:, 0::2] = c & 15
    out[:, 1::2] = c >> 4
    return out


CASES = [
    # B, H, W, C, O, R, S, stride, pad, G, bits, out_bits
    (2, 9, 7, 16, 24, 3, 3, 1, 1, 4, 8, 8),
    (3, 8, 8, 64, 100, 3, 3, 1, 1, 64, 8, 4),
    (3, 8, 8, 64, 100, 3, 3, 2, 1, 64, 4, 8),
    (2, 15, 15, 4, 16, 7, 7, 2, 3, 4, 8, 4),
    (2, 12, 12, 32, 64, 1, 1, 2, 0, 8, 4, 4),
    (2, 6, 6, 6, 6, 3, 3, 1, 1, 3, 8, 8),       # direct path only (C % 4 != 0)
    (32, 28, 28, 128, 128, 3, 3, 1, 1, 4, 8, 8),  # benchmark layer, G=4
    (32, 28, 28, 128, 128, 3, 3, 1, 1, 64, 8, 8),  # and G=64
    (2, 9, 11, 256, 72, 3, 3, 1, 1, 4, 4, 4),   # input-patch staging, two chunks
]


@pytest.mark.parametrize("prepared_path", [True, False], ids=["matrix-core", "direct"])
@pytest.mark.parametrize("case", CASES)
def test_fused_quantization(case, prepared_path):
    B, H, W, C, O, R, S, st, pd, G, bits, out_bits = case
    w = fi.he_weights(O, C, R, S, "fused", case)
    x = fi.relu_gauss((B, H, W, C), "fused", case)
    codes, alpha, _ = fgq.fgq_ternarize(dev(w), G)
    q, sx = fgq.fgq_quantize_act(dev(x), bits)
    K = R * S * C
    prep = fgq.fgq_prepare_weights(codes, alpha, O, K, G) if prepared_path else None
    y = fgq.fgq_conv2d(q, bits, sx, (B, H, W, C), codes, alpha, O, R, S, st, pd, G, prepared=prep)
    qmax = 255 if out_bits == 8 else 15
    yh = host(y).reshape(-1, O)
    s_out = np.float32(0.9 * float(np.max(yh)) / qmax)   # some outputs clip at qmax
    sc = dev(np.array([s_out], np.float32))
    q_fused = host(fgq.fgq_conv2d_q(q, bits, sx, (B, H, W, C), codes, alpha, O, R, S, st, pd, G, out_bits,
                                    sc, prepared=prep)).ravel()
    q_two, _ = fgq.fgq_quantize_act(y.reshape(-1), out_bits, scale_in=sc)
    np.testing.assert_array_equal(q_fused, host(q_two))

    # against the oracle on sampled rows
    t, a, _ = oracle.ternarize(w, G)
    codes_ref = oracle.pack_codes(t)
    q_ref, s_ref = oracle.quantize_act(x, bits)
    M = yh.shape[0]
    n = min(M, 160)
    got = unpack(q_fused, out_bits, O)
    for row0 in sorted({0, M - n}):
        y_ref = oracle.conv2d(q_ref, bits, s_ref, x.shape, codes_ref, a, O, R, S, (st, st), (pd, pd), G,
                              rows=(row0, n))[row0:row0 + n]
        c_ref = unpack(oracle.quantize_act(y_ref.ravel(), out_bits, s_out)[0], out_bits, O)
        diff = got[row0:row0 + n] - c_ref
        if not prepared_path:
            assert not diff.any()
            continue
        P = oracle.group_sums_conv(q_ref, bits, x.shape, codes_ref, O, R, S, (st, st), (pd, pd), G,
                                   row0, n).astype(np.float64)
        mag = float(s_ref) * np.einsum("mog,og->mo", np.abs(P), a.astype(np.float64))
        u = y_ref.astype(np.float64) / float(s_out)
        near = np.abs(u - np.floor(u) - 0.5) <= (TOL * mag + 2 * np.abs(y_ref) * 2.0 ** -24) / float(s_out)
        assert np.all(np.abs(diff) <= 1), "codes differ by more than one step"
        assert not (diff != 0)[~near].any(), f"{int(((diff != 0) & ~near).sum())} codes differ away from a tie"


@pytest.mark.parametrize("out_bits", [8, 4])
def test_fused_gemm(out_bits):
    M, K, O, G = 77, 256, 128, 4
    w = fi.gauss_weights(O, K, 0.05, "fused-gemm")
    x = fi.relu_gauss((M, K), "fused-gemm")
    codes, alpha, _ = fgq.fgq_ternarize(dev(w), G)
    q, sx = fgq.fgq_quantize_act(dev(x), 8)
    prep = fgq.fgq_prepare_weights(codes, alpha, O, K, G)
    y = fgq.fgq_gemm(q, 8, sx, M, K, codes, alpha, O, G, prepared=prep)
    sc = dev(np.array([np.float32(float(host(y).max()) / (2 ** out_bits - 1))], np.float32))
    q_fused = fgq.fgq_gemm_q(q, 8, sx, M, K, codes, alpha, O, G, out_bits, sc, prepared=prep)
    q_two, _ = fgq.fgq_quantize_act(y.reshape(-1), out_bits, scale_in=sc)
    np.testing.assert_array_equal(host(q_fused).ravel(), host(q_two))
