"""GEMMs with split K (fully-connected layers at small batch), through the C
ABI: fgq_gemm_ws must equal fgq_gemm / fgq_gemm_q bit for bit (same integer
totals, same epilogue), and fgq_gemm_dfp_ws must equal the oracle bit for
bit; every case below is one where the split is taken (workspace size > 0).
"""
import ctypes

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


CASES = [
    # M, K, O, G, bits
    (5, 4096, 96, 4, 8),
    (64, 2048, 1000, 4, 8),
    (3, 1024, 64, 8, 4),
    (4, 1000, 96, 4, 8),          # K not a multiple of the 128-wide step
    (64, 9216, 512, 4, 8),        # AlexNet fc6 reduction length
    (1, 4096, 1000, 2, 8),        # a single row
]


def setup(M, K, O, G, bits, tag):
    # These tests compare kernels with each other on layers the folded layout
    # accepts: magnitudes below 0.1 sigma are raised to it, which keeps every
    # group scale within a small factor of its channel's largest (scales
    # near zero fail the layout's accuracy guard; test_gpu_guard.py covers
    # that route).
    w = fi.gauss_weights(O, K, 0.02, "splitk", tag)
    w = np.where(w < 0, -1.0, 1.0).astype(np.float32) * np.maximum(np.abs(w), np.float32(0.002))
    x = fi.relu_gauss((M, K), "splitk", tag)
    codes, alpha, _ = fgq.fgq_ternarize(dev(w), G)
    q, sx = fgq.fgq_quantize_act(dev(x), bits)
    return w, x, codes, alpha, q, sx


def oracle_close(w, x, y, M, K, O, G, bits):
    """y within 1e-5 of the oracle's summand magnitude, element by element."""
    t, a, _ = oracle.ternarize(w, G)
    qr, sr = oracle.quantize_act(x, bits)
    y_ref, mag = oracle.conv2d_rows(qr, bits, sr, (1, M, 1, K), oracle.pack_codes(t), a, O, 1, 1, (1, 1),
                                    (0, 0), G, np.arange(M))
    err = np.abs(y.reshape(M, O).astype(np.float64) - y_ref.astype(np.float64))
    assert np.all(err <= 1e-5 * mag), f"worst {np.max(err / np.maximum(mag, 1e-300)):.3e}"


@pytest.mark.parametrize("case", CASES)
def test_gemm_ws_equals_unsplit(case):
    M, K, O, G, bits = case
    assert fgq.fgq_gemm_ws_bytes(M, K, O, G) > 0
    w, x, codes, alpha, q, sx = setup(*case, tag=case)
    prep = fgq.fgq_prepare_weights(codes, alpha, O, K, G)
    y = host(fgq.fgq_gemm(q, bits, sx, M, K, codes, alpha, O, G, prepared=prep))
    y_ws = host(fgq.fgq_gemm_ws(q, bits, sx, M, K, codes, alpha, O, G, prepared=prep))
    np.testing.assert_array_equal(y_ws.view(np.uint32), y.view(np.uint32))
    oracle_close(w, x, y_ws, M, K, O, G, bits)
    for out_bits in (8, 4):
        sc = dev(np.array([np.float32(0.9 * float(np.abs(y).max()) / (2 ** out_bits - 1))], np.float32))
        a = host(fgq.fgq_gemm_q(q, bits, sx, M, K, codes, alpha, O, G, out_bits, sc, prepared=prep))
        b = host(fgq.fgq_gemm_ws(q, bits, sx, M, K, codes, alpha, O, G, prepared=prep, out_bits=out_bits,
                                 out_scale=sc))
        np.testing.assert_array_equal(a.ravel(), b.ravel())


@pytest.mark.parametrize("case", CASES)
def test_gemm_dfp_ws_bit_exact(case):
    M, K, O, G, bits = case
    assert fgq.fgq_gemm_ws_bytes(M, K, O, G, fixed_point=True) > 0
    w, x, codes, alpha, q, sx = setup(*case, tag=("dfp", case))
    prep = fgq.fgq_prepare_weights_dfp(codes, alpha, O, K, G, 8)
    y = host(fgq.fgq_gemm_dfp_ws(q, bits, sx, M, K, codes, prep, O, G))
    t, a, _ = oracle.ternarize(w, G)
    qr, sr = oracle.quantize_act(x, bits)
    A, fl = oracle.dfp_alpha(a, 8)
    y_ref = oracle.gemm_dfp(qr, bits, sr, M, K, oracle.pack_codes(t), A, fl, O, G)
    np.testing.assert_array_equal(y.view(np.uint32), y_ref.view(np.uint32))
    s_out = np.float32(0.8 * float(np.abs(y_ref).max()) / 255)
    got = host(fgq.fgq_gemm_dfp_ws(q, bits, sx, M, K, codes, prep, O, G, out_bits=8,
                                   out_scale=dev(np.array([s_out], np.float32)))).ravel()
    np.testing.assert_array_equal(got, oracle.quantize_act(y_ref.ravel(), 8, s_out)[0])


# Shapes of the codes-expanding kernel (M <= 64, K % 64 == 0, G a power of
# two in 4..128): one or two 32-row blocks, every scale-code width, a K tail
# of half a step, channels that do not fill the last 128-wide tile, 4-bit
# activations, and long K (many splits of up to 8 steps).
DFPX_CASES = [
    # M, K, O, G, bits
    (64, 9216, 256, 4, 8),
    (1, 9216, 384, 4, 8),
    (32, 2048, 200, 8, 8),
    (33, 4160, 128, 16, 8),       # K % 128 == 64
    (7, 4096, 160, 32, 4),
    (40, 4160, 96, 64, 4),        # K % 128 == 64, 4-bit
    (64, 4096, 130, 128, 8),
    (2, 1024, 64, 4, 4),
]


@pytest.mark.parametrize("case", DFPX_CASES)
def test_gemm_dfp_ws_codes_path(case):
    M, K, O, G, bits = case
    w, x, codes, alpha, q, sx = setup(*case, tag=("dfpx", case))
    prep = fgq.fgq_prepare_weights_dfp(codes, alpha, O, K, G, 8)
    t, a, _ = oracle.ternarize(w, G)
    qr, sr = oracle.quantize_act(x, bits)
    A, fl = oracle.dfp_alpha(a, 8)
    y_ref = oracle.gemm_dfp(qr, bits, sr, M, K, oracle.pack_codes(t), A, fl, O, G)
    y = host(fgq.fgq_gemm_dfp_ws(q, bits, sx, M, K, codes, prep, O, G))
    np.testing.assert_array_equal(y.view(np.uint32), y_ref.view(np.uint32))
    for out_bits in (8, 4):
        s_out = np.float32(0.8 * float(np.abs(y_ref).max()) / (2 ** out_bits - 1))
        got = host(fgq.fgq_gemm_dfp_ws(q, bits, sx, M, K, codes, prep, O, G, out_bits=out_bits,
                                       out_scale=dev(np.array([s_out], np.float32)))).ravel()
        ref = oracle.quantize_act(y_ref.ravel(), out_bits, s_out)[0]
        np.testing.assert_array_equal(got, ref)


@pytest.mark.parametrize("case", DFPX_CASES)
def test_gemm_ws_codes_path_equals_unsplit(case):
    # fp32 scales: the expanding kernel on the folded layout (three digit
    # planes) must give the unsplit kernel's integer sums and epilogue
    M, K, O, G, bits = case
    w, x, codes, alpha, q, sx = setup(*case, tag=("x3", case))
    prep = fgq.fgq_prepare_weights(codes, alpha, O, K, G)
    y = host(fgq.fgq_gemm(q, bits, sx, M, K, codes, alpha, O, G, prepared=prep))
    y_ws = host(fgq.fgq_gemm_ws(q, bits, sx, M, K, codes, alpha, O, G, prepared=prep))
    np.testing.assert_array_equal(y_ws.view(np.uint32), y.view(np.uint32))
    oracle_close(w, x, y_ws, M, K, O, G, bits)
    sc = dev(np.array([np.float32(0.9 * float(np.abs(y).max()) / 255)], np.float32))
    a = host(fgq.fgq_gemm_q(q, bits, sx, M, K, codes, alpha, O, G, 8, sc, prepared=prep))
    b = host(fgq.fgq_gemm_ws(q, bits, sx, M, K, codes, alpha, O, G, prepared=prep, out_bits=8, out_scale=sc))
    np.testing.assert_array_equal(a.ravel(), b.ravel())


@pytest.mark.parametrize("fixed_point", [True, False])
def test_codes_path_with_unaligned_workspace(fixed_point):
    # a workspace 4-byte but not 16-byte aligned: sums leave from registers
    M, K, O, G, bits = 48, 2048, 256, 4, 8
    w, x, codes, alpha, q, sx = setup(M, K, O, G, bits, tag=("ua", fixed_point))
    nb = fgq.fgq_gemm_ws_bytes(M, K, O, G, fixed_point)
    big = torch.empty(nb + 16, dtype=torch.uint8, device="cuda")
    ws = big[4:4 + nb]
    assert ws.data_ptr() % 16 == 4
    if fixed_point:
        prep = fgq.fgq_prepare_weights_dfp(codes, alpha, O, K, G, 8)
        ref = host(fgq.fgq_gemm_dfp(q, bits, sx, M, K, codes, prep, O, G))
        got = host(fgq.fgq_gemm_dfp_ws(q, bits, sx, M, K, codes, prep, O, G, ws=ws))
    else:
        prep = fgq.fgq_prepare_weights(codes, alpha, O, K, G)
        ref = host(fgq.fgq_gemm(q, bits, sx, M, K, codes, alpha, O, G, prepared=prep))
        got = host(fgq.fgq_gemm_ws(q, bits, sx, M, K, codes, alpha, O, G, prepared=prep, ws=ws))
    np.testing.assert_array_equal(got.view(np.uint32), ref.view(np.uint32))


def test_gemm_ws_missing_workspace_and_no_split():
    M, K, O, G, bits = CASES[0]
    w, x, codes, alpha, q, sx = setup(M, K, O, G, bits, "ws")
    prep = fgq.fgq_prepare_weights(codes, alpha, O, K, G)
    y = torch.empty((M, O), dtype=torch.float32, device="cuda")
    L = fgq.lib()
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    ptr = lambda t: ctypes.c_void_p(t.data_ptr())
    rc = L.fgq_gemm_ws(ptr(q), bits, ptr(sx), M, K, ptr(codes), ptr(alpha), ptr(prep), O, G, 0, None, ptr(y),
                       None, 0, stream)
    assert rc == 8
    small = torch.empty(16, dtype=torch.uint8, device="cuda")
    rc = L.fgq_gemm_ws(ptr(q), bits, ptr(sx), M, K, ptr(codes), ptr(alpha), ptr(prep), O, G, 0, None, ptr(y),
                       ptr(small), 16, stream)
    assert rc == 8
    # a shape that fills the device needs no workspace and equals fgq_gemm
    M2, K2, O2 = 640, 256, 128
    assert fgq.fgq_gemm_ws_bytes(M2, K2, O2, 4) == 0
    w, x, codes, alpha, q, sx = setup(M2, K2, O2, 4, 8, "ws2")
    prep = fgq.fgq_prepare_weights(codes, alpha, O2, K2, 4)
    a = host(fgq.fgq_gemm(q, 8, sx, M2, K2, codes, alpha, O2, 4, prepared=prep))
    b = host(fgq.fgq_gemm_ws(q, 8, sx, M2, K2, codes, alpha, O2, 4, prepared=prep))
    np.testing.assert_array_equal(a.view(np.uint32), b.view(np.uint32))
