"""The largest reduction length of the int8 matrix-core kernels, at the
int32 extreme, against the oracle through the C ABI.

The folded (three-plane), one-plane fixed-point and codes-expanding kernels
accumulate in int32 and accept K <= 65536: 255 * 127 * 65536 < 2^31 is the
largest sum they can meet (every activation at 255, every weight code at
+/-127).  One step past the limit the folded GEMM must fall back to the
direct kernel and stay exact.  Cases: all-maximal activations with
equal-magnitude weights (every group kept whole, so every scale is the
common magnitude and every fixed-point code is 127), and random ones.
"""
import numpy as np
import pytest
import torch

import fgq_inputs as fi
import oracle

fgq = pytest.importorskip("paper_1705_01462_amd")

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

KMAX = 65536


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def layer(M, K, O, extreme, tag):
    """extreme: "max" (every product +255*127: the int32 bound itself),
    "signs" (equal magnitudes, random signs) or None (random layer)."""
    if extreme:
        sign = np.ones((O, K)) if extreme == "max" else \
            np.where(fi.rng("lim-sign", K, O, tag).random((O, K)) < 0.5, -1.0, 1.0)
        w = (0.9921875 * sign).astype(np.float32)  # 127/128: fixed-point code 127
        x = np.ones((M, K), np.float32)
    else:
        w = fi.gauss_weights(O, K, 0.01, "lim", K, O, tag)
        x = fi.relu_gauss((M, K), "lim", K, tag)
    return w, x


def summand_mag(q, sx, t, alpha, G):
    qd = q.astype(np.float64)
    M, K = qd.shape
    O = t.shape[0]
    ng = K // G
    P = np.abs(np.einsum("mgi,ogi->mog", qd.reshape(M, ng, G), t.astype(np.float64).reshape(O, ng, G)))
    return float(sx) * np.einsum("mog,og->mo", P, alpha.astype(np.float64))


@pytest.mark.parametrize("extreme", ["max", "signs", None])
def test_folded_gemm_at_max_k(extreme):
    M, K, O, G = 3, KMAX, 32, 4
    w, x = layer(M, K, O, extreme, "fold")
    codes, alpha, _ = fgq.fgq_ternarize(dev(w), G)
    q, sx = fgq.fgq_quantize_act(dev(x.ravel()), 8)
    prep = fgq.fgq_prepare_weights(codes, alpha, O, K, G)
    y = host(fgq.fgq_gemm(q, 8, sx, M, K, codes, alpha, O, G, prepared=prep))
    t, a, _ = oracle.ternarize(w, G)
    qr, sr = oracle.quantize_act(x, 8)
    y_ref = oracle.gemm(qr, 8, sr, M, K, oracle.pack_codes(t), a, O, G)
    if extreme:
        assert np.all(qr == 255) and np.all(np.abs(t) == 1)
    mag = summand_mag(qr.reshape(M, K), sr, t, a, G)
    assert np.all(np.abs(y.astype(np.float64) - y_ref) <= 1e-5 * mag)
    # the codes-expanding kernel (split K) gives the same integer sums
    y_ws = host(fgq.fgq_gemm_ws(q, 8, sx, M, K, codes, alpha, O, G, prepared=prep))
    np.testing.assert_array_equal(y_ws.view(np.uint32), y.view(np.uint32))


def test_folded_gemm_past_max_k_falls_back_exact():
    M, K, O, G = 2, KMAX + 128, 32, 4
    w, x = layer(M, K, O, "signs", "past")
    codes, alpha, _ = fgq.fgq_ternarize(dev(w), G)
    q, sx = fgq.fgq_quantize_act(dev(x.ravel()), 8)
    prep = fgq.fgq_prepare_weights(codes, alpha, O, K, G)
    y = host(fgq.fgq_gemm(q, 8, sx, M, K, codes, alpha, O, G, prepared=prep))
    t, a, _ = oracle.ternarize(w, G)
    qr, sr = oracle.quantize_act(x, 8)
    y_ref = oracle.gemm(qr, 8, sr, M, K, oracle.pack_codes(t), a, O, G)
    np.testing.assert_array_equal(y.view(np.uint32), y_ref.view(np.uint32))


@pytest.mark.parametrize("M", [64, 2])
@pytest.mark.parametrize("extreme", ["max", "signs", None])
def test_fixed_point_gemm_at_max_k(M, extreme):
    K, O, G = KMAX, 128, 4
    w, x = layer(M, K, O, extreme, ("dfp", M))
    codes, alpha, _ = fgq.fgq_ternarize(dev(w), G)
    q, sx = fgq.fgq_quantize_act(dev(x.ravel()), 8)
    prep = fgq.fgq_prepare_weights_dfp(codes, alpha, O, K, G, 8)
    t, a, _ = oracle.ternarize(w, G)
    qr, sr = oracle.quantize_act(x, 8)
    A, fl = oracle.dfp_alpha(a, 8)
    if extreme:
        assert np.all(A == 127)
    y_ref = oracle.gemm_dfp(qr, 8, sr, M, K, oracle.pack_codes(t), A, fl, O, G)
    # one-plane kernel, then the codes-expanding kernel with split K
    y1 = host(fgq.fgq_gemm_dfp(q, 8, sx, M, K, codes, prep, O, G))
    np.testing.assert_array_equal(y1.view(np.uint32), y_ref.view(np.uint32))
    y2 = host(fgq.fgq_gemm_dfp_ws(q, 8, sx, M, K, codes, prep, O, G))
    np.testing.assert_array_equal(y2.view(np.uint32), y_ref.view(np.uint32))
