"""Python (numpy + ctypes) front end of the CPU oracle for FGQ inference.

TEST INFRASTRUCTURE ONLY: imported by tests/, by __graft_entry__.smoke() and
by the CPU-baseline leg of bench.py, never by the library package.  Every
function here marshals numpy arrays into the plain C oracle (fgq_oracle.c);
the arithmetic lives there.  Conventions are documented in fgq_oracle.h.
"""
import ctypes
import os

import numpy as np

from . import build as _build

EXACT = 0       # Eq. (5) solved by exhaustive threshold search
EXP_LEMMA = 1   # Lemma 1: Delta = mean |W|
GAUSS = 3       # Gaussian-optimal threshold 0.612 * rms(W)
KS = 4          # per layer: EXP_LEMMA or GAUSS, by the K-S test (Sec. 3.1)

_lib = None

_c_i32 = ctypes.c_int32
_c_i64 = ctypes.c_int64
_c_f32 = ctypes.c_float
_c_p = ctypes.c_void_p


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_build.LIB):
            _build.build()
        L = ctypes.CDLL(_build.LIB)
        L.orc_ternarize_group.argtypes = [_c_p, _c_i64, _c_i64, ctypes.c_int, _c_p, _c_i64, _c_p, _c_p]
        L.orc_ternarize.argtypes = [_c_p, _c_i64, _c_i64, _c_i32, _c_i32, _c_i32, _c_i32, _c_p, _c_p, _c_p]
        L.orc_pack_codes.argtypes = [_c_p, _c_i64, _c_i64, _c_p]
        L.orc_pack_codes.restype = None
        L.orc_unpack_codes.argtypes = [_c_p, _c_i64, _c_i64, _c_p]
        L.orc_unpack_codes.restype = None
        L.orc_quantize_act.argtypes = [_c_p, _c_i64, _c_i32, _c_p, _c_p, _c_p]
        L.orc_group_sums_conv.argtypes = [_c_p, _c_i32, _c_i64, _c_i64, _c_i64, _c_i64, _c_p, _c_i64,
                                          _c_i32, _c_i32, _c_i32, _c_i32, _c_i32, _c_i32, _c_i32,
                                          _c_i64, _c_i64, _c_p]
        L.orc_conv2d.argtypes = [_c_p, _c_i32, _c_f32, _c_i64, _c_i64, _c_i64, _c_i64, _c_p, _c_p,
                                 _c_i64, _c_i32, _c_i32, _c_i32, _c_i32, _c_i32, _c_i32, _c_i32,
                                 _c_i64, _c_i64, _c_i32, _c_p]
        L.orc_gemm.argtypes = [_c_p, _c_i32, _c_f32, _c_i64, _c_i64, _c_p, _c_p, _c_i64, _c_i32,
                               _c_i32, _c_p]
        L.orc_conv2d_rows.argtypes = [_c_p, _c_i32, _c_f32, _c_i64, _c_i64, _c_i64, _c_i64, _c_p, _c_p,
                                      _c_i64, _c_i32, _c_i32, _c_i32, _c_i32, _c_i32, _c_i32, _c_i32,
                                      _c_p, _c_i64, _c_i32, _c_p, _c_p]
        L.orc_dfp_alpha.argtypes = [_c_p, _c_i64, _c_i32, _c_p, _c_p]
        L.orc_conv2d_dfp.argtypes = [_c_p, _c_i32, _c_f32, _c_i64, _c_i64, _c_i64, _c_i64, _c_p, _c_p,
                                     _c_i32, _c_i64, _c_i32, _c_i32, _c_i32, _c_i32, _c_i32, _c_i32,
                                     _c_i32, _c_i64, _c_i64, _c_i32, _c_p]
        L.orc_gemm_dfp.argtypes = [_c_p, _c_i32, _c_f32, _c_i64, _c_i64, _c_p, _c_p, _c_i32, _c_i64,
                                   _c_i32, _c_i32, _c_p]
        L.orc_w8_quantize.argtypes = [_c_p, _c_i64, _c_p, _c_p]
        L.orc_conv2d_w8.argtypes = [_c_p, _c_i32, _c_f32, _c_i64, _c_i64, _c_i64, _c_i64, _c_p, _c_i32,
                                    _c_i64, _c_i32, _c_i32, _c_i32, _c_i32, _c_i32, _c_i32, _c_i64,
                                    _c_i64, _c_i32, _c_p]
        L.orc_max_threads.argtypes = []
        L.orc_ternarize_group_asym.argtypes = [_c_p, _c_i64, _c_i64, _c_p, _c_i64, _c_p, _c_p, _c_p]
        L.orc_ternarize_asym.argtypes = [_c_p, _c_i64, _c_i64, _c_i32, _c_i32, _c_i32, _c_p, _c_p, _c_p, _c_p]
        L.orc_ks_distances.argtypes = [_c_p, _c_i64, _c_p]
        L.orc_gauss_u.argtypes = []
        L.orc_gauss_u.restype = ctypes.c_double
        for f in ("orc_ternarize_group", "orc_ternarize", "orc_quantize_act",
                  "orc_group_sums_conv", "orc_conv2d", "orc_conv2d_rows", "orc_gemm", "orc_dfp_alpha",
                  "orc_conv2d_dfp", "orc_gemm_dfp", "orc_w8_quantize", "orc_conv2d_w8",
                  "orc_max_threads", "orc_ternarize_group_asym", "orc_ternarize_asym",
                  "orc_ks_distances"):
            getattr(L, f).restype = ctypes.c_int
        _lib = L
    return _lib


class OracleError(RuntimeError):
    def __init__(self, code):
        super().__init__(f"oracle returned status {code}")
        self.code = code


def _check(rc):
    if rc != 0:
        raise OracleError(rc)


def _ptr(a):
    return a.ctypes.data_as(ctypes.c_void_p)


def ternarize_group(w, method=EXACT):
    """One group: returns (t int8[n], alpha float32, delta float32)."""
    w = np.ascontiguousarray(w, dtype=np.float32).ravel()
    t = np.zeros(w.size, np.int8)
    a = np.zeros(1, np.float32)
    d = np.zeros(1, np.float32)
    _check(lib().orc_ternarize_group(_ptr(w), w.size, 1, method, _ptr(t), 1, _ptr(a), _ptr(d)))
    return t, a[0], d[0]


def ternarize(w, G, method=EXACT):
    """Layer weights float32 [O][C][R][S] (a 2-D [O][K] array is a 1x1 conv).

    Returns t int8 [O][K] (k = (r*S+s)*C + c), alpha and delta float32 [O][K/G].
    """
    w = np.ascontiguousarray(w, dtype=np.float32)
    if w.ndim == 2:
        w = w.reshape(w.shape[0], w.shape[1], 1, 1)
    O, C, R, S = w.shape
    K = C * R * S
    t = np.zeros((O, K), np.int8)
    a = np.zeros((O, K // G if G > 0 and K % G == 0 else 1), np.float32)
    d = np.zeros_like(a)
    _check(lib().orc_ternarize(_ptr(w), O, C, R, S, G, method, _ptr(t), _ptr(a), _ptr(d)))
    return t, a, d


def ternarize_group_asym(w):
    """One group, Eq. (3)-(4): returns (t int8[n], alpha, delta_p, delta_n)."""
    w = np.ascontiguousarray(w, dtype=np.float32).ravel()
    t = np.zeros(w.size, np.int8)
    a, dp, dn = (np.zeros(1, np.float32) for _ in range(3))
    _check(lib().orc_ternarize_group_asym(_ptr(w), w.size, 1, _ptr(t), 1, _ptr(a), _ptr(dp), _ptr(dn)))
    return t, a[0], dp[0], dn[0]


def ternarize_asym(w, G):
    """Layer weights as for ternarize; returns t, alpha, delta_p, delta_n."""
    w = np.ascontiguousarray(w, dtype=np.float32)
    if w.ndim == 2:
        w = w.reshape(w.shape[0], w.shape[1], 1, 1)
    O, C, R, S = w.shape
    K = C * R * S
    t = np.zeros((O, K), np.int8)
    a = np.zeros((O, K // G if G > 0 and K % G == 0 else 1), np.float32)
    dp, dn = np.zeros_like(a), np.zeros_like(a)
    _check(lib().orc_ternarize_asym(_ptr(w), O, C, R, S, G, _ptr(t), _ptr(a), _ptr(dp), _ptr(dn)))
    return t, a, dp, dn


def ks_distances(w):
    """K-S distances of |w| (storage order) to the fitted half-normal and
    exponential laws: returns (d_gauss, d_exp)."""
    w = np.ascontiguousarray(w, dtype=np.float32).ravel()
    d = np.zeros(2, np.float64)
    _check(lib().orc_ks_distances(_ptr(w), w.size, _ptr(d)))
    return float(d[0]), float(d[1])


def gauss_u():
    return float(lib().orc_gauss_u())


KS_SAMPLE = 16384


def paper_weight_layout(w, N):
    """Sec. 3.2's weight layout [K][C/N][R*S][N] of weights [O][C][R][S] (the
    paper's K is the output-channel count, O here): for each output channel,
    input-channel block and filter tap, the N weights of one group are
    contiguous.  A pure rearrangement (no arithmetic)."""
    w = np.asarray(w)
    O, C, R, S = w.shape
    if C % N:
        raise ValueError("N must divide C")
    return np.ascontiguousarray(w.reshape(O, C // N, N, R * S).transpose(0, 1, 3, 2))


def pack_codes(t):
    t = np.ascontiguousarray(t, dtype=np.int8)
    O, K = t.shape
    codes = np.zeros((O, (K + 3) // 4), np.uint8)
    lib().orc_pack_codes(_ptr(t), O, K, _ptr(codes))
    return codes


def unpack_codes(codes, K):
    codes = np.ascontiguousarray(codes, dtype=np.uint8)
    O = codes.shape[0]
    t = np.zeros((O, K), np.int8)
    lib().orc_unpack_codes(_ptr(codes), O, K, _ptr(t))
    return t


def quantize_act(x, bits, scale=None):
    """Returns (q packed uint8, scale float32)."""
    x = np.ascontiguousarray(x, dtype=np.float32).ravel()
    nbytes = x.size if bits == 8 else x.size // 2
    q = np.zeros(max(nbytes, 1), np.uint8)
    s_out = np.zeros(1, np.float32)
    s_in = None if scale is None else np.array([scale], np.float32)
    _check(lib().orc_quantize_act(_ptr(x), x.size, bits, None if s_in is None else _ptr(s_in),
                                  _ptr(q), _ptr(s_out)))
    return q[:nbytes], s_out[0]


def conv_out_hw(H, W, R, S, stride, pad):
    return (H + 2 * pad[0] - R) // stride[0] + 1, (W + 2 * pad[1] - S) // stride[1] + 1


def group_sums_conv(q, bits, shape, codes, O, R, S, stride, pad, G, row0=0, nrows=None):
    """Exact int32 group sums P[rows][O][K/G] of a conv; shape = (B, H, W, C)."""
    B, H, W, C = shape
    Ho, Wo = conv_out_hw(H, W, R, S, stride, pad)
    M = B * Ho * Wo
    if nrows is None:
        nrows = M - row0
    K = R * S * C
    P = np.zeros((nrows, O, K // G), np.int32)
    q = np.ascontiguousarray(q, dtype=np.uint8)
    codes = np.ascontiguousarray(codes, dtype=np.uint8)
    _check(lib().orc_group_sums_conv(_ptr(q), bits, B, H, W, C, _ptr(codes), O, R, S,
                                     stride[0], stride[1], pad[0], pad[1], G, row0, nrows,
                                     _ptr(P)))
    return P


def conv2d(q, bits, sx, shape, codes, alpha, O, R, S, stride, pad, G, rows=None, nthreads=0):
    """fp32 output [B*Ho*Wo][O].  rows=(row0, nrows) restricts the rows computed
    (other rows are left NaN)."""
    B, H, W, C = shape
    Ho, Wo = conv_out_hw(H, W, R, S, stride, pad)
    M = B * Ho * Wo
    y = np.full((M, O), np.nan, np.float32)
    row0, nrows = (0, -1) if rows is None else rows
    q = np.ascontiguousarray(q, dtype=np.uint8)
    codes = np.ascontiguousarray(codes, dtype=np.uint8)
    alpha = np.ascontiguousarray(alpha, dtype=np.float32)
    _check(lib().orc_conv2d(_ptr(q), bits, float(sx), B, H, W, C, _ptr(codes), _ptr(alpha), O,
                            R, S, stride[0], stride[1], pad[0], pad[1], G, row0, nrows,
                            nthreads, _ptr(y)))
    return y


def conv2d_rows(q, bits, sx, shape, codes, alpha, O, R, S, stride, pad, G, rows, nthreads=0):
    """The layer on the listed output rows: (y float32 [len(rows)][O], summand
    magnitude s_x * sum_g alpha_g |P_g| float64 [len(rows)][O])."""
    B, H, W, C = shape
    rows = np.ascontiguousarray(rows, dtype=np.int64)
    y = np.empty((len(rows), O), np.float32)
    mag = np.empty((len(rows), O), np.float64)
    q = np.ascontiguousarray(q, dtype=np.uint8)
    codes = np.ascontiguousarray(codes, dtype=np.uint8)
    alpha = np.ascontiguousarray(alpha, dtype=np.float32)
    _check(lib().orc_conv2d_rows(_ptr(q), bits, float(sx), B, H, W, C, _ptr(codes), _ptr(alpha), O,
                                 R, S, stride[0], stride[1], pad[0], pad[1], G, _ptr(rows), len(rows),
                                 nthreads, _ptr(y), _ptr(mag)))
    return y, mag


def gemm(q, bits, sx, M, K, codes, alpha, O, G, nthreads=0):
    y = np.zeros((M, O), np.float32)
    q = np.ascontiguousarray(q, dtype=np.uint8)
    codes = np.ascontiguousarray(codes, dtype=np.uint8)
    alpha = np.ascontiguousarray(alpha, dtype=np.float32)
    _check(lib().orc_gemm(_ptr(q), bits, float(sx), M, K, _ptr(codes), _ptr(alpha), O, G,
                          nthreads, _ptr(y)))
    return y


def dfp_alpha(alpha, bits):
    """Sec. 4 fixed-point group scales: returns (A int8, same shape as alpha; fl)."""
    alpha = np.ascontiguousarray(alpha, dtype=np.float32)
    A = np.zeros(alpha.shape, np.int8)
    fl = np.zeros(1, np.int32)
    _check(lib().orc_dfp_alpha(_ptr(alpha), alpha.size, bits, _ptr(A), _ptr(fl)))
    return A, int(fl[0])


def conv2d_dfp(q, bits, sx, shape, codes, A, fl, O, R, S, stride, pad, G, rows=None, nthreads=0):
    """fp32 output [B*Ho*Wo][O] of the fixed-point-scale layer; rows as in conv2d."""
    B, H, W, C = shape
    Ho, Wo = conv_out_hw(H, W, R, S, stride, pad)
    M = B * Ho * Wo
    y = np.full((M, O), np.nan, np.float32)
    row0, nrows = (0, -1) if rows is None else rows
    q = np.ascontiguousarray(q, dtype=np.uint8)
    codes = np.ascontiguousarray(codes, dtype=np.uint8)
    A = np.ascontiguousarray(A, dtype=np.int8)
    _check(lib().orc_conv2d_dfp(_ptr(q), bits, float(sx), B, H, W, C, _ptr(codes), _ptr(A), fl, O,
                                R, S, stride[0], stride[1], pad[0], pad[1], G, row0, nrows,
                                nthreads, _ptr(y)))
    return y


def gemm_dfp(q, bits, sx, M, K, codes, A, fl, O, G, nthreads=0):
    y = np.zeros((M, O), np.float32)
    q = np.ascontiguousarray(q, dtype=np.uint8)
    codes = np.ascontiguousarray(codes, dtype=np.uint8)
    A = np.ascontiguousarray(A, dtype=np.int8)
    _check(lib().orc_gemm_dfp(_ptr(q), bits, float(sx), M, K, _ptr(codes), _ptr(A), fl, O, G,
                              nthreads, _ptr(y)))
    return y


def w8_quantize(w):
    """First layer at 8-bit weights: returns (W8 int8, same shape as w; fl)."""
    w = np.ascontiguousarray(w, dtype=np.float32)
    W8 = np.zeros(w.shape, np.int8)
    fl = np.zeros(1, np.int32)
    _check(lib().orc_w8_quantize(_ptr(w), w.size, _ptr(W8), _ptr(fl)))
    return W8, int(fl[0])


def conv2d_w8(q, bits, sx, shape, W8, fl, O, R, S, stride, pad, rows=None, nthreads=0):
    """fp32 output [B*Ho*Wo][O] of the 8-bit-weight layer; W8 is [O][C][R][S]."""
    B, H, W, C = shape
    Ho, Wo = conv_out_hw(H, W, R, S, stride, pad)
    M = B * Ho * Wo
    y = np.full((M, O), np.nan, np.float32)
    row0, nrows = (0, -1) if rows is None else rows
    q = np.ascontiguousarray(q, dtype=np.uint8)
    W8 = np.ascontiguousarray(W8, dtype=np.int8)
    _check(lib().orc_conv2d_w8(_ptr(q), bits, float(sx), B, H, W, C, _ptr(W8), fl, O, R, S,
                               stride[0], stride[1], pad[0], pad[1], row0, nrows, nthreads, _ptr(y)))
    return y


def max_threads():
    return lib().orc_max_threads()
