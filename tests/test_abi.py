"""The C ABI of libfgq.so, checked without a GPU: the library loads, exports
every entry point include/fgq.h declares, and rejects invalid arguments on
the host before anything is enqueued."""
import ctypes
import os
import re

import pytest

import paper_1705_01462_amd as fgq

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "fgq.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(fgq_[a-z0-9_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    names = declared_functions()
    assert "fgq_conv2d" in names and "fgq_ternarize" in names and len(names) >= 13
    L = ctypes.CDLL(fgq.LIB_PATH)
    for n in names:
        assert hasattr(L, n), n
    # the binding wraps every entry point under the same name
    for n in ("fgq_ternarize", "fgq_quantize_act", "fgq_prepare_weights", "fgq_conv2d",
              "fgq_gemm", "fgq_group_sums", "fgq_conv2d_q", "fgq_gemm_q", "fgq_dfp_alpha",
              "fgq_prepare_weights_dfp", "fgq_conv2d_dfp", "fgq_gemm_dfp",
              "fgq_prepare_weights_w8", "fgq_conv2d_w8", "fgq_gemm_ws", "fgq_gemm_dfp_ws"):
        assert callable(getattr(fgq, n))


def test_checking_build_exports_every_declared_symbol():
    """libfgq_check.so (the -DFGQ_CHECK build) has the same ABI; the normal
    library answers fgq_check_violations with FGQ_ERR_UNSUPPORTED."""
    path = os.path.join(os.path.dirname(fgq.LIB_PATH), "libfgq_check.so")
    if not os.path.exists(path):
        pytest.skip("checking build not built")
    L = ctypes.CDLL(path)
    for n in declared_functions():
        assert hasattr(L, n), n
    N = ctypes.CDLL(os.path.join(os.path.dirname(fgq.LIB_PATH), "libfgq.so"))
    N.fgq_check_violations.argtypes = [ctypes.c_void_p] * 3
    n = ctypes.c_int64(-1)
    assert N.fgq_check_violations(ctypes.byref(n), None, None) == 7
    L.fgq_check_violations.argtypes = [ctypes.c_void_p] * 3
    assert L.fgq_check_violations(None, None, None) == 1  # FGQ_ERR_NULL before any device call


def test_host_helpers():
    L = fgq.lib()
    assert L.fgq_abi_version() == 2
    assert L.fgq_codes_bytes(128, 1152) == 128 * 288
    assert L.fgq_codes_bytes(3, 5) == 3 * 2
    assert L.fgq_group_count(128, 1152, 4) == 128 * 288
    assert L.fgq_group_count(128, 1152, 5) == -1
    assert L.fgq_prepared_bytes(128, 1152, 4) >= 3 * 128 * 1152
    assert L.fgq_prepared_bytes(128, 1152, 5) == 0
    assert L.fgq_prepared_bytes(128, 1152, 4) % 256 == 0
    assert L.fgq_quantize_ws_bytes(32 * 28 * 28 * 128) >= 4
    for code in range(10):
        assert L.fgq_status_string(code).startswith(b"FGQ")
    # per-group layout (G = 64, at most 160 groups): 2-bit codes + alpha
    assert L.fgq_prepared_bytes(128, 1152, 64) == 128 * 1152 // 4 + 4 * 18 * 128
    assert L.fgq_prepared_bytes(40, 64 * 161, 64) >= 3 * 64 * 64 * 161  # folded beyond 160 groups


# Arguments that fail validation are rejected before any HIP call, so these
# use placeholder pointers.  Skip them where a device exists, so that a
# validation bug could never launch a kernel on bogus addresses.
no_device = pytest.mark.skipif(fgq.lib().fgq_device_count() > 0,
                               reason="placeholder pointers are only passed on a host without a GPU")
P = ctypes.c_void_p(0x1000)
N = None


@no_device
def test_ternarize_validation():
    L = fgq.lib()
    assert L.fgq_ternarize(N, 4, 8, 3, 3, 4, 0, P, P, P, N) == 1
    assert L.fgq_ternarize(P, 0, 8, 3, 3, 4, 0, P, P, P, N) == 2
    assert L.fgq_ternarize(P, 4, 8, 3, 3, 3, 0, P, P, P, N) == 3
    assert L.fgq_ternarize(P, 4, 8, 3, 3, 4, 7, P, P, P, N) == 7


@no_device
def test_probe_validation():
    L = fgq.lib()
    assert L.fgq_probe_mfma_i8(4, 8, N, 1024, N) == 1
    assert L.fgq_probe_mfma_i8(0, 8, P, 1024, N) == 2
    assert L.fgq_probe_mfma_i8(4, 0, P, 1024, N) == 2
    assert L.fgq_probe_mfma_i8(4, 8, P, 1023, N) == 2   # needs blocks * 256 sink elements


@no_device
def test_quantize_validation():
    L = fgq.lib()
    assert L.fgq_quantize_act(N, 16, 8, N, P, P, P, 4096, N) == 1
    assert L.fgq_quantize_act(P, 16, 6, N, P, P, P, 4096, N) == 4
    assert L.fgq_quantize_act(P, 15, 4, N, P, P, P, 4096, N) == 4
    assert L.fgq_quantize_act(P, 0, 8, N, P, P, P, 4096, N) == 2
    assert L.fgq_quantize_act(P, 16, 8, N, P, P, N, 0, N) == 8   # dynamic scale needs ws


@no_device
def test_fused_layer_validation():
    L = fgq.lib()
    args = lambda O, ob, sc, qo: (P, 8, P, 2, 8, 8, 16, P, P, None, O, 3, 3, 1, 1, 1, 1, 4, ob, sc, qo, None)
    assert L.fgq_conv2d_q(*args(16, 7, P, P)) == 4          # FGQ_ERR_BITS: out_bits
    assert L.fgq_conv2d_q(*args(15, 4, P, P)) == 4          # 4-bit output needs even O
    assert L.fgq_conv2d_q(*args(16, 8, None, P)) == 1       # FGQ_ERR_NULL: scale
    assert L.fgq_conv2d_q(*args(16, 8, P, None)) == 1       # FGQ_ERR_NULL: q_out
    assert L.fgq_gemm_q(P, 8, P, 4, 16, P, P, None, 15, 4, 4, P, P, None) == 4


def test_prepared_bytes_dfp():
    L = fgq.lib()
    # header 256, one int8 plane O32*Kp, bias 4*O, dequantized scales 4*O*K/G,
    # then for the codes-expanding GEMM the 2-bit codes (O128*Kp/4) and the
    # scale codes (O128*Kp/64 * 64/G) in its operand order (each region
    # 256-byte aligned)
    plane = 128 * 1152
    bias_off = 256 + plane
    alpha_off = bias_off + 512
    xcodes_off = alpha_off + 4 * 128 * 288
    xacodes_off = xcodes_off + 128 * 1152 // 4
    assert L.fgq_prepared_bytes_dfp(128, 1152, 4) == xacodes_off + 128 * 1152 // 4
    # G = 64: one scale-code byte per lane and 128-wide step
    assert L.fgq_prepared_bytes_dfp(128, 1152, 64) == (alpha_off + 4 * 128 * 18 + 255) // 256 * 256 \
        + 128 * 1152 // 4 + 128 * 1152 // 64
    assert L.fgq_prepared_bytes_dfp(128, 1152, 5) == 0
    # O padded to 32, K to 128
    assert L.fgq_prepared_bytes_dfp(33, 100, 4) % 256 == 0
    assert L.fgq_prepared_bytes_dfp(33, 100, 4) >= 256 + 64 * 128 + 4 * 33 + 5 * 33 * 25


@no_device
def test_dfp_validation():
    L = fgq.lib()
    assert L.fgq_dfp_alpha(None, 4, 8, P, P, None) == 1
    assert L.fgq_dfp_alpha(P, 4, 6, P, P, None) == 4
    assert L.fgq_dfp_alpha(P, 0, 8, P, P, None) == 2
    assert L.fgq_prepare_weights_dfp(P, P, 16, 64, 4, 6, P, 1 << 20, None) == 4   # alpha bits
    assert L.fgq_prepare_weights_dfp(P, P, 16, 64, 3, 8, P, 1 << 20, None) == 3   # G
    assert L.fgq_prepare_weights_dfp(P, P, 16, 64, 4, 8, P, 16, None) == 8        # too small
    conv = lambda ob, O, sc, prep: L.fgq_conv2d_dfp(P, 8, P, 2, 8, 8, 16, P, prep, O, 3, 3, 1, 1,
                                                    1, 1, 4, ob, sc, P, None)
    assert conv(7, 16, P, P) == 4                                  # out_bits
    assert conv(4, 15, P, P) == 4                                  # 4-bit output needs even O
    assert conv(8, 16, None, P) == 1                               # scale for codes
    assert conv(0, 16, None, None) == 1                            # prepared required
    assert conv(0, 16, None, ctypes.c_void_p(0x1001)) == 8         # prepared alignment
    assert L.fgq_gemm_dfp(P, 8, P, 4, 16, P, P, 16, 5, 0, None, P, None) == 3


def test_gemm_ws_bytes():
    L = fgq.lib()
    # no device here: 256 compute units assumed.  fc6 at batch 64: 32 channel
    # tiles of 128; splits capped so the int32 sums stay within a quarter of
    # the weight bytes: min(512/32, 72/2, 9216/(16*64)) = 9 -> 8 steps each, 9 splits
    assert L.fgq_gemm_ws_bytes(64, 9216, 4096, 4, 0) == 9 * 3 * 64 * 4096 * 4
    assert L.fgq_gemm_ws_bytes(64, 9216, 4096, 4, 1) == 9 * 1 * 64 * 4096 * 4
    # the codes-expanding GEMM (M <= 64, K % 16 == 0, G a power of two in
    # 4..128) always writes sums per split: splits of up to 8 steps
    assert L.fgq_gemm_ws_bytes(64, 256, 128, 4, 0) == 1 * 3 * 64 * 128 * 4
    assert L.fgq_gemm_ws_bytes(64, 256, 128, 4, 1) == 1 * 1 * 64 * 128 * 4
    assert L.fgq_gemm_ws_bytes(64, 264, 128, 4, 0) == 0          # K % 16 != 0, too few steps
    assert L.fgq_gemm_ws_bytes(65, 256, 128, 4, 0) == 0          # M > 64, too few steps
    assert L.fgq_gemm_ws_bytes(64, 9216, 4096, 64, 0) == 0        # per-group layout: no split
    assert L.fgq_gemm_ws_bytes(64, 9216, 4096, 64, 1) > 0
    assert L.fgq_gemm_ws_bytes(64, 9216, 4096, 5, 0) == 0         # G does not divide K


def test_prepared_bytes_w8():
    L = fgq.lib()
    # the fixed-point layout with one group per tap: header, plane, bias, R*S scales per channel
    assert L.fgq_prepared_bytes_w8(64, 4, 7, 7) == L.fgq_prepared_bytes_dfp(64, 196, 4)
    assert L.fgq_prepared_bytes_w8(0, 4, 7, 7) == 0


@no_device
def test_w8_validation():
    L = fgq.lib()
    assert L.fgq_prepare_weights_w8(None, 64, 4, 7, 7, P, 1 << 20, None) == 1
    assert L.fgq_prepare_weights_w8(P, 64, 4, 7, 7, P, 16, None) == 8
    assert L.fgq_prepare_weights_w8(P, 64, 0, 7, 7, P, 1 << 20, None) == 2
    conv = lambda ob, sc: L.fgq_conv2d_w8(P, 8, P, 2, 8, 8, 16, P, 16, 3, 3, 1, 1, 1, 1, ob, sc, P, None)
    assert conv(5, P) == 4
    assert conv(8, None) == 1


@no_device
def test_layer_validation():
    L = fgq.lib()
    conv = L.fgq_conv2d
    ok = dict(B=2, H=8, W=8, C=16, O=8, R=3, S=3, sh=1, sw=1, ph=1, pw=1, G=4)

    def call(bits=8, q=P, prepared=N, **kw):
        a = dict(ok, **kw)
        return conv(q, bits, P, a["B"], a["H"], a["W"], a["C"], P, P, prepared, a["O"], a["R"],
                    a["S"], a["sh"], a["sw"], a["ph"], a["pw"], a["G"], P, N)

    assert call(q=N) == 1
    assert call(bits=5) == 4
    assert call(bits=4, C=15, G=5) == 4
    assert call(G=3) == 3
    assert call(G=0) == 3
    assert call(B=0) == 2
    assert call(sh=0) == 2
    assert call(ph=-1) == 2
    assert call(H=1, ph=0) == 2                    # kernel larger than the padded image
    assert call(prepared=ctypes.c_void_p(0x1001)) == 8   # misaligned prepared buffer
    assert L.fgq_gemm(P, 8, P, 4, 64, P, P, N, 8, 3, P, N) == 3
    assert L.fgq_group_sums(P, 8, 2, 8, 8, 16, P, 8, 3, 3, 1, 1, 1, 1, 4, 0, 129, P, N) == 2
    assert L.fgq_group_sums(P, 8, 2, 8, 8, 16, P, 8, 3, 3, 1, 1, 1, 1, 4, -1, 1, P, N) == 2
    assert L.fgq_prepare_weights(P, P, 8, 64, 4, ctypes.c_void_p(0x1010), 1 << 20, N) == 8
    assert L.fgq_prepare_weights(P, P, 8, 64, 4, P, 16, N) == 8
    assert L.fgq_prepare_weights(P, P, 8, 64, 3, P, 1 << 20, N) == 3


@no_device
def test_no_device_reports_hip_error():
    assert fgq.lib().fgq_device_count() == 0


@no_device
def test_residual_validation():
    L = fgq.lib()
    geo = (P, 8, P, 2, 8, 8, 16, P, P, None, 16, 3, 3, 1, 1, 1, 1, 4)
    assert L.fgq_conv2d_residual(*geo, None, P, None) == 1              # FGQ_ERR_NULL: res
    assert L.fgq_conv2d_residual(*geo, P, None, None) == 1              # FGQ_ERR_NULL: y
    assert L.fgq_conv2d_residual(P, 8, P, 2, 8, 8, 15, P, P, None, 16, 3, 3, 1, 1, 1, 1, 4,
                                 P, P, None) == 3                       # FGQ_ERR_GROUP: C % G
    rq = lambda O, ob, sc, qo: L.fgq_conv2d_residual_q(P, 8, P, 2, 8, 8, 16, P, P, None, O, 3, 3, 1, 1, 1, 1,
                                                       4, P, P, ob, sc, qo, None)
    assert rq(16, 7, P, P) == 4                                         # out_bits
    assert rq(15, 4, P, P) == 4                                         # 4-bit output needs even O
    assert rq(16, 8, None, P) == 1                                      # scale for codes
    assert rq(16, 8, P, None) == 1                                      # q_out
    dr = lambda ob, sc, qo, prep: L.fgq_conv2d_dfp_residual(P, 8, P, 2, 8, 8, 16, P, prep, 16, 3, 3, 1, 1, 1, 1,
                                                            4, P, P, ob, sc, qo, None)
    assert dr(0, None, None, None) == 1                                 # prepared required
    assert dr(8, None, P, P) == 1                                       # scale for codes
    assert dr(8, P, None, P) == 1                                       # q_out for codes
    assert dr(6, P, P, P) == 4                                          # out_bits
    assert dr(0, None, None, ctypes.c_void_p(0x1001)) == 8              # prepared alignment
