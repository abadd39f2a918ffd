"""Python binding of libfgq.so (FGQ ternary inference on MI355X / gfx950).

Thin ctypes marshalling over the C ABI declared in include/fgq.h: every
function below has the name of the C entry point it calls, checks device,
dtype and contiguity, allocates outputs with torch (device memory only) and
passes raw pointers plus torch's current HIP stream.  No arithmetic of the
method happens here; there is no CPU fallback -- if the library is missing,
importing the call raises.
"""
import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
# FGQ_LIBRARY=check selects the checking build, libfgq_check.so (bounds-
# checked loads and stores, fgq_check_violations), in place of libfgq.so.
LIB_PATH = os.path.join(_HERE, "libfgq_check.so" if os.environ.get("FGQ_LIBRARY") == "check" else "libfgq.so")

FGQ_TERN_EXACT = 0
FGQ_TERN_EXP_LEMMA = 1
FGQ_TERN_GAUSS = 3
FGQ_TERN_KS = 4

_STATUS = {0: "FGQ_OK", 1: "FGQ_ERR_NULL", 2: "FGQ_ERR_SHAPE", 3: "FGQ_ERR_GROUP",
           4: "FGQ_ERR_BITS", 5: "FGQ_ERR_NONFINITE", 6: "FGQ_ERR_HIP",
           7: "FGQ_ERR_UNSUPPORTED", 8: "FGQ_ERR_WORKSPACE", 9: "FGQ_ERR_RANGE"}
FGQ_ERR_RANGE = 9


class FgqError(RuntimeError):
    def __init__(self, code, where):
        super().__init__(f"{where}: {_STATUS.get(code, code)}")
        self.code = code


_lib = None
_P = ctypes.c_void_p
_I32 = ctypes.c_int32
_I64 = ctypes.c_int64
_SZ = ctypes.c_size_t

_SIGS = {
    "fgq_status_string": ([_I32], ctypes.c_char_p),
    "fgq_abi_version": ([], _I32),
    "fgq_check_violations": ([_P, _P, _P], _I32),
    "fgq_device_count": ([], _I32),
    "fgq_codes_bytes": ([_I64, _I64], _SZ),
    "fgq_group_count": ([_I64, _I64, _I32], _I64),
    "fgq_ternarize": ([_P, _I64, _I64, _I32, _I32, _I32, _I32, _P, _P, _P, _P], _I32),
    "fgq_ternarize_asym": ([_P, _I64, _I64, _I32, _I32, _I32, _P, _P, _P, _P, _P], _I32),
    "fgq_ks_distances": ([_P, _I64, _P, _P], _I32),
    "fgq_quantize_ws_bytes": ([_I64], _SZ),
    "fgq_quantize_act": ([_P, _I64, _I32, _P, _P, _P, _P, _SZ, _P], _I32),
    "fgq_quantize_act_noalloc": ([_P, _I64, _I32, _P, _P, _P, _P], _I32),
    "fgq_prepared_bytes": ([_I64, _I64, _I32], _SZ),
    "fgq_prepare_weights": ([_P, _P, _I64, _I64, _I32, _P, _SZ, _P], _I32),
    "fgq_conv2d": ([_P, _I32, _P, _I64, _I64, _I64, _I64, _P, _P, _P, _I64, _I32, _I32,
                    _I32, _I32, _I32, _I32, _I32, _P, _P], _I32),
    "fgq_conv2d_residual": ([_P, _I32, _P, _I64, _I64, _I64, _I64, _P, _P, _P, _I64, _I32, _I32,
                             _I32, _I32, _I32, _I32, _I32, _P, _P, _P], _I32),
    "fgq_conv2d_residual_q": ([_P, _I32, _P, _I64, _I64, _I64, _I64, _P, _P, _P, _I64, _I32, _I32,
                               _I32, _I32, _I32, _I32, _I32, _P, _P, _I32, _P, _P, _P], _I32),
    "fgq_conv2d_dfp_residual": ([_P, _I32, _P, _I64, _I64, _I64, _I64, _P, _P, _I64, _I32, _I32,
                                 _I32, _I32, _I32, _I32, _I32, _P, _P, _I32, _P, _P, _P], _I32),
    "fgq_gemm": ([_P, _I32, _P, _I64, _I64, _P, _P, _P, _I64, _I32, _P, _P], _I32),
    "fgq_conv2d_q": ([_P, _I32, _P, _I64, _I64, _I64, _I64, _P, _P, _P, _I64, _I32, _I32,
                      _I32, _I32, _I32, _I32, _I32, _I32, _P, _P, _P], _I32),
    "fgq_gemm_q": ([_P, _I32, _P, _I64, _I64, _P, _P, _P, _I64, _I32, _I32, _P, _P, _P], _I32),
    "fgq_group_sums": ([_P, _I32, _I64, _I64, _I64, _I64, _P, _I64, _I32, _I32, _I32, _I32,
                        _I32, _I32, _I32, _I64, _I64, _P, _P], _I32),
    "fgq_dfp_alpha": ([_P, _I64, _I32, _P, _P, _P], _I32),
    "fgq_prepared_bytes_dfp": ([_I64, _I64, _I32], _SZ),
    "fgq_prepare_weights_dfp": ([_P, _P, _I64, _I64, _I32, _I32, _P, _SZ, _P], _I32),
    "fgq_conv2d_dfp": ([_P, _I32, _P, _I64, _I64, _I64, _I64, _P, _P, _I64, _I32, _I32, _I32,
                        _I32, _I32, _I32, _I32, _I32, _P, _P, _P], _I32),
    "fgq_gemm_dfp": ([_P, _I32, _P, _I64, _I64, _P, _P, _I64, _I32, _I32, _P, _P, _P], _I32),
    "fgq_gemm_ws_bytes": ([_I64, _I64, _I64, _I32, _I32], _SZ),
    "fgq_gemm_ws": ([_P, _I32, _P, _I64, _I64, _P, _P, _P, _I64, _I32, _I32, _P, _P, _P, _SZ, _P], _I32),
    "fgq_gemm_dfp_ws": ([_P, _I32, _P, _I64, _I64, _P, _P, _I64, _I32, _I32, _P, _P, _P, _SZ, _P], _I32),
    "fgq_prepared_bytes_w8": ([_I64, _I64, _I32, _I32], _SZ),
    "fgq_prepare_weights_w8": ([_P, _I64, _I64, _I32, _I32, _P, _SZ, _P], _I32),
    "fgq_conv2d_w8": ([_P, _I32, _P, _I64, _I64, _I64, _I64, _P, _I64, _I32, _I32, _I32, _I32,
                       _I32, _I32, _I32, _P, _P, _P], _I32),
    "fgq_probe_mfma_i8": ([_I32, _I32, _P, _I64, _P], _I32),
}


def lib():
    """The loaded libfgq.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{os.path.basename(LIB_PATH)} not found at {LIB_PATH}; run "
                               "__graft_entry__.build() (hipcc --offload-arch=gfx950) first")
        L = ctypes.CDLL(LIB_PATH)
        for name, (args, res) in _SIGS.items():
            f = getattr(L, name)
            f.argtypes = args
            f.restype = res
        _lib = L
    return _lib


def _check(rc, where):
    if rc != 0:
        raise FgqError(rc, where)


def fgq_check_violations():
    """Checking build only: (count, first_site, first_offset) of the
    suppressed out-of-bounds accesses since the previous call (cleared)."""
    n, site, off = ctypes.c_int64(0), ctypes.c_int32(0), ctypes.c_int64(0)
    _check(lib().fgq_check_violations(ctypes.byref(n), ctypes.byref(site), ctypes.byref(off)),
           "fgq_check_violations")
    return n.value, site.value, off.value


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _dev(t, dtype, name):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be a GPU tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def conv_out_hw(H, W, R, S, stride, pad):
    return (H + 2 * pad[0] - R) // stride[0] + 1, (W + 2 * pad[1] - S) // stride[1] + 1


def _pair(v):
    return (v, v) if isinstance(v, int) else tuple(v)


def fgq_ternarize(w, G, method=FGQ_TERN_EXACT, want_delta=True):
    """w: fp32 [O][C][R][S] (or [O][K]).  Returns (codes uint8 [O][ceil(K/4)],
    alpha fp32 [O][K/G], delta fp32 [O][K/G] or None)."""
    w4 = w if w.dim() == 4 else w.reshape(w.shape[0], w.shape[1], 1, 1)
    O, C, R, S = w4.shape
    K = C * R * S
    pw = _dev(w4, torch.float32, "w")
    codes = torch.empty((O, (K + 3) // 4), dtype=torch.uint8, device=w.device)
    ng = K // G if G > 0 and K % G == 0 else 1
    alpha = torch.empty((O, ng), dtype=torch.float32, device=w.device)
    delta = torch.empty_like(alpha) if want_delta else None
    rc = lib().fgq_ternarize(pw, O, C, R, S, G, method, codes.data_ptr(), alpha.data_ptr(),
                             delta.data_ptr() if delta is not None else None, _stream())
    _check(rc, "fgq_ternarize")
    return codes, alpha, delta


def fgq_ternarize_asym(w, G):
    """Eq. (3)-(4) per group.  Returns (codes, alpha, delta_p, delta_n)."""
    w4 = w if w.dim() == 4 else w.reshape(w.shape[0], w.shape[1], 1, 1)
    O, C, R, S = w4.shape
    K = C * R * S
    pw = _dev(w4, torch.float32, "w")
    codes = torch.empty((O, (K + 3) // 4), dtype=torch.uint8, device=w.device)
    ng = K // G if G > 0 and K % G == 0 else 1
    alpha = torch.empty((O, ng), dtype=torch.float32, device=w.device)
    dp, dn = torch.empty_like(alpha), torch.empty_like(alpha)
    rc = lib().fgq_ternarize_asym(pw, O, C, R, S, G, codes.data_ptr(), alpha.data_ptr(), dp.data_ptr(),
                                  dn.data_ptr(), _stream())
    _check(rc, "fgq_ternarize_asym")
    return codes, alpha, dp, dn


def fgq_ks_distances(w):
    """K-S distances of |w| to the fitted half-normal and exponential laws:
    a device fp64 tensor [D_gauss, D_exp]."""
    pw = _dev(w, torch.float32, "w")
    d = torch.empty(2, dtype=torch.float64, device=w.device)
    _check(lib().fgq_ks_distances(pw, w.numel(), d.data_ptr(), _stream()), "fgq_ks_distances")
    return d


def fgq_quantize_ws_bytes(n):
    return int(lib().fgq_quantize_ws_bytes(n))


def fgq_quantize_act(x, bits, scale_in=None, q=None, scale_out=None, ws=None):
    """x: fp32 tensor (any shape, contiguous).  Returns (q uint8 packed, scale fp32[1])."""
    n = x.numel()
    px = _dev(x, torch.float32, "x")
    nbytes = n if bits == 8 else n // 2
    if q is None:
        q = torch.empty(max(nbytes, 1), dtype=torch.uint8, device=x.device)[:nbytes]
    if scale_out is None:
        scale_out = torch.empty(1, dtype=torch.float32, device=x.device)
    if scale_in is None and ws is None:
        ws = torch.empty(max(fgq_quantize_ws_bytes(n), 4), dtype=torch.uint8, device=x.device)
    rc = lib().fgq_quantize_act(px, n, bits,
                                None if scale_in is None else _dev(scale_in, torch.float32, "scale_in"),
                                _dev(q, torch.uint8, "q"), _dev(scale_out, torch.float32, "scale_out"),
                                None if ws is None else ctypes.c_void_p(ws.data_ptr()),
                                0 if ws is None else ws.numel() * ws.element_size(), _stream())
    _check(rc, "fgq_quantize_act")
    return q, scale_out


def fgq_quantize_act_noalloc(x, bits, scale_in=None, q=None, scale_out=None):
    """fgq_quantize_act without a workspace (the library's per-device scratch);
    allocates nothing when q and scale_out are given."""
    n = x.numel()
    px = _dev(x, torch.float32, "x")
    nbytes = n if bits == 8 else n // 2
    if q is None:
        q = torch.empty(max(nbytes, 1), dtype=torch.uint8, device=x.device)[:nbytes]
    if scale_out is None:
        scale_out = torch.empty(1, dtype=torch.float32, device=x.device)
    rc = lib().fgq_quantize_act_noalloc(px, n, bits,
                                        None if scale_in is None else _dev(scale_in, torch.float32, "scale_in"),
                                        _dev(q, torch.uint8, "q"), _dev(scale_out, torch.float32, "scale_out"),
                                        _stream())
    _check(rc, "fgq_quantize_act_noalloc")
    return q, scale_out


def fgq_prepared_bytes(O, K, G):
    return int(lib().fgq_prepared_bytes(O, K, G))


def fgq_prepare_weights(codes, alpha, O, K, G, prepared=None, fallback=False):
    """Per-layer constants of the matrix-core kernels (opaque uint8 buffer).

    When the folded layout cannot meet its accuracy bound for some channel
    (FGQ_ERR_RANGE: the channel's group scales spread too widely), raises
    FgqError, or with fallback=True returns None, so that the layer calls
    given prepared=None run the direct kernel."""
    nb = fgq_prepared_bytes(O, K, G)
    if nb == 0:
        raise FgqError(3, "fgq_prepare_weights")
    if prepared is None:
        prepared = torch.empty(nb, dtype=torch.uint8, device=codes.device)
    if prepared.data_ptr() % 256:
        raise ValueError("prepared buffer must be 256-byte aligned")
    rc = lib().fgq_prepare_weights(_dev(codes, torch.uint8, "codes"), _dev(alpha, torch.float32, "alpha"),
                                   O, K, G, ctypes.c_void_p(prepared.data_ptr()), nb, _stream())
    if rc == FGQ_ERR_RANGE and fallback:
        return None
    _check(rc, "fgq_prepare_weights")
    return prepared


def fgq_conv2d(q, bits, sx, shape, codes, alpha, O, R, S, stride, pad, G, prepared=None, y=None):
    """q: NHWC activations (packed uint8); shape = (B, H, W, C); sx: fp32[1]
    device scalar.  Returns y fp32 [B][Ho][Wo][O]."""
    B, H, W, C = shape
    sh, sw = _pair(stride)
    ph, pw = _pair(pad)
    Ho, Wo = conv_out_hw(H, W, R, S, (sh, sw), (ph, pw))
    if y is None:
        y = torch.empty((B, Ho, Wo, O), dtype=torch.float32, device=q.device)
    rc = lib().fgq_conv2d(_dev(q, torch.uint8, "q"), bits, _dev(sx, torch.float32, "sx"), B, H, W, C,
                          _dev(codes, torch.uint8, "codes"), _dev(alpha, torch.float32, "alpha"),
                          None if prepared is None else _dev(prepared, torch.uint8, "prepared"),
                          O, R, S, sh, sw, ph, pw, G, _dev(y, torch.float32, "y"), _stream())
    _check(rc, "fgq_conv2d")
    return y


def fgq_conv2d_residual(q, bits, sx, shape, codes, alpha, O, R, S, stride, pad, G, res, prepared=None, y=None):
    """fgq_conv2d with a residual block's shortcut addition and ReLU fused:
    y = max(conv + res, 0), res fp32 [B][Ho][Wo][O] (y may be res itself)."""
    B, H, W, C = shape
    sh, sw = _pair(stride)
    ph, pw = _pair(pad)
    Ho, Wo = conv_out_hw(H, W, R, S, (sh, sw), (ph, pw))
    if y is None:
        y = torch.empty((B, Ho, Wo, O), dtype=torch.float32, device=q.device)
    for t, name in ((res, "res"), (y, "y")):
        if isinstance(t, torch.Tensor) and t.numel() != B * Ho * Wo * O:
            raise ValueError(f"{name} must hold B*Ho*Wo*O = {B * Ho * Wo * O} values, got {t.numel()}")
    rc = lib().fgq_conv2d_residual(_dev(q, torch.uint8, "q"), bits, _dev(sx, torch.float32, "sx"), B, H, W, C,
                                   _dev(codes, torch.uint8, "codes"), _dev(alpha, torch.float32, "alpha"),
                                   None if prepared is None else _dev(prepared, torch.uint8, "prepared"),
                                   O, R, S, sh, sw, ph, pw, G, _dev(res, torch.float32, "res"),
                                   _dev(y, torch.float32, "y"), _stream())
    _check(rc, "fgq_conv2d_residual")
    return y


def fgq_conv2d_residual_q(q, bits, sx, shape, codes, alpha, O, R, S, stride, pad, G, res, out_bits, out_scale,
                          prepared=None, y=None, q_out=None):
    """fgq_conv2d_residual that also writes the codes of its output at the
    device scale out_scale (fp32[1]): returns (y, q_out)."""
    B, H, W, C = shape
    sh, sw = _pair(stride)
    ph, pw = _pair(pad)
    Ho, Wo = conv_out_hw(H, W, R, S, (sh, sw), (ph, pw))
    n = B * Ho * Wo * O
    if y is None:
        y = torch.empty((B, Ho, Wo, O), dtype=torch.float32, device=q.device)
    if q_out is None:
        q_out = torch.empty((B, Ho, Wo, O * out_bits // 8), dtype=torch.uint8, device=q.device)
    for t, name, want in ((res, "res", n), (y, "y", n), (q_out, "q_out", n * out_bits // 8)):
        if isinstance(t, torch.Tensor) and t.numel() != want:
            raise ValueError(f"{name} must hold {want} values, got {t.numel()}")
    rc = lib().fgq_conv2d_residual_q(_dev(q, torch.uint8, "q"), bits, _dev(sx, torch.float32, "sx"), B, H, W, C,
                                     _dev(codes, torch.uint8, "codes"), _dev(alpha, torch.float32, "alpha"),
                                     None if prepared is None else _dev(prepared, torch.uint8, "prepared"),
                                     O, R, S, sh, sw, ph, pw, G, _dev(res, torch.float32, "res"),
                                     _dev(y, torch.float32, "y"), out_bits,
                                     _dev(out_scale, torch.float32, "out_scale"), _dev(q_out, torch.uint8, "q_out"),
                                     _stream())
    _check(rc, "fgq_conv2d_residual_q")
    return y, q_out


def fgq_gemm(q, bits, sx, M, K, codes, alpha, O, G, prepared=None, y=None):
    if y is None:
        y = torch.empty((M, O), dtype=torch.float32, device=q.device)
    rc = lib().fgq_gemm(_dev(q, torch.uint8, "q"), bits, _dev(sx, torch.float32, "sx"), M, K,
                        _dev(codes, torch.uint8, "codes"), _dev(alpha, torch.float32, "alpha"),
                        None if prepared is None else _dev(prepared, torch.uint8, "prepared"),
                        O, G, _dev(y, torch.float32, "y"), _stream())
    _check(rc, "fgq_gemm")
    return y


def fgq_conv2d_q(q, bits, sx, shape, codes, alpha, O, R, S, stride, pad, G, out_bits, out_scale,
                 prepared=None, q_out=None):
    """fgq_conv2d with the next layer's quantization fused: returns uint8
    codes NHWC [B][Ho][Wo][O] (out_bits 8) or [B][Ho][Wo][O/2] (out_bits 4)
    with the device scale out_scale (fp32[1])."""
    B, H, W, C = shape
    sh, sw = _pair(stride)
    ph, pw = _pair(pad)
    Ho, Wo = conv_out_hw(H, W, R, S, (sh, sw), (ph, pw))
    if q_out is None:
        q_out = torch.empty((B, Ho, Wo, O * out_bits // 8), dtype=torch.uint8, device=q.device)
    rc = lib().fgq_conv2d_q(_dev(q, torch.uint8, "q"), bits, _dev(sx, torch.float32, "sx"), B, H, W, C,
                            _dev(codes, torch.uint8, "codes"), _dev(alpha, torch.float32, "alpha"),
                            None if prepared is None else _dev(prepared, torch.uint8, "prepared"),
                            O, R, S, sh, sw, ph, pw, G, out_bits, _dev(out_scale, torch.float32, "out_scale"),
                            _dev(q_out, torch.uint8, "q_out"), _stream())
    _check(rc, "fgq_conv2d_q")
    return q_out


def fgq_gemm_q(q, bits, sx, M, K, codes, alpha, O, G, out_bits, out_scale, prepared=None, q_out=None):
    if q_out is None:
        q_out = torch.empty((M, O * out_bits // 8), dtype=torch.uint8, device=q.device)
    rc = lib().fgq_gemm_q(_dev(q, torch.uint8, "q"), bits, _dev(sx, torch.float32, "sx"), M, K,
                          _dev(codes, torch.uint8, "codes"), _dev(alpha, torch.float32, "alpha"),
                          None if prepared is None else _dev(prepared, torch.uint8, "prepared"),
                          O, G, out_bits, _dev(out_scale, torch.float32, "out_scale"),
                          _dev(q_out, torch.uint8, "q_out"), _stream())
    _check(rc, "fgq_gemm_q")
    return q_out


def fgq_dfp_alpha(alpha, bits, A=None, fl=None):
    """Fixed-point group scales (one fractional length per layer): returns
    (A int8 tensor shaped like alpha, fl int32[1] device scalar)."""
    if A is None:
        A = torch.empty(alpha.shape, dtype=torch.int8, device=alpha.device)
    if fl is None:
        fl = torch.empty(1, dtype=torch.int32, device=alpha.device)
    rc = lib().fgq_dfp_alpha(_dev(alpha, torch.float32, "alpha"), alpha.numel(), bits,
                             _dev(A, torch.int8, "A"), _dev(fl, torch.int32, "fl"), _stream())
    _check(rc, "fgq_dfp_alpha")
    return A, fl


def fgq_prepared_bytes_dfp(O, K, G):
    return int(lib().fgq_prepared_bytes_dfp(O, K, G))


def fgq_prepare_weights_dfp(codes, alpha, O, K, G, alpha_bits, prepared=None):
    """Constants of the layer with fixed-point scales (opaque uint8 buffer)."""
    nb = fgq_prepared_bytes_dfp(O, K, G)
    if nb == 0:
        raise FgqError(3, "fgq_prepare_weights_dfp")
    if prepared is None:
        prepared = torch.empty(nb, dtype=torch.uint8, device=codes.device)
    if prepared.data_ptr() % 256:
        raise ValueError("prepared buffer must be 256-byte aligned")
    rc = lib().fgq_prepare_weights_dfp(_dev(codes, torch.uint8, "codes"), _dev(alpha, torch.float32, "alpha"),
                                       O, K, G, alpha_bits, ctypes.c_void_p(prepared.data_ptr()), nb,
                                       _stream())
    _check(rc, "fgq_prepare_weights_dfp")
    return prepared


def _dfp_out(shape_rows, O, out_bits, device, out):
    if out is not None:
        return out
    if out_bits == 0:
        return torch.empty(shape_rows + (O,), dtype=torch.float32, device=device)
    return torch.empty(shape_rows + (O * out_bits // 8,), dtype=torch.uint8, device=device)


def fgq_conv2d_dfp(q, bits, sx, shape, codes, prepared, O, R, S, stride, pad, G, out_bits=0,
                   out_scale=None, out=None):
    """The layer with fixed-point scales: fp32 y [B][Ho][Wo][O] (out_bits 0)
    or the next layer's codes (out_bits 8 or 4, with out_scale)."""
    B, H, W, C = shape
    sh, sw = _pair(stride)
    ph, pw = _pair(pad)
    Ho, Wo = conv_out_hw(H, W, R, S, (sh, sw), (ph, pw))
    out = _dfp_out((B, Ho, Wo), O, out_bits, q.device, out)
    rc = lib().fgq_conv2d_dfp(_dev(q, torch.uint8, "q"), bits, _dev(sx, torch.float32, "sx"), B, H, W, C,
                              _dev(codes, torch.uint8, "codes"), _dev(prepared, torch.uint8, "prepared"),
                              O, R, S, sh, sw, ph, pw, G, out_bits,
                              None if out_scale is None else _dev(out_scale, torch.float32, "out_scale"),
                              ctypes.c_void_p(out.data_ptr()), _stream())
    _check(rc, "fgq_conv2d_dfp")
    return out


def fgq_gemm_dfp(q, bits, sx, M, K, codes, prepared, O, G, out_bits=0, out_scale=None, out=None):
    out = _dfp_out((M,), O, out_bits, q.device, out)
    rc = lib().fgq_gemm_dfp(_dev(q, torch.uint8, "q"), bits, _dev(sx, torch.float32, "sx"), M, K,
                            _dev(codes, torch.uint8, "codes"), _dev(prepared, torch.uint8, "prepared"),
                            O, G, out_bits,
                            None if out_scale is None else _dev(out_scale, torch.float32, "out_scale"),
                            ctypes.c_void_p(out.data_ptr()), _stream())
    _check(rc, "fgq_gemm_dfp")
    return out


def fgq_gemm_ws_bytes(M, K, O, G, fixed_point=False):
    return int(lib().fgq_gemm_ws_bytes(M, K, O, G, 1 if fixed_point else 0))


def _ws_for(M, K, O, G, fixed_point, device, ws):
    nb = fgq_gemm_ws_bytes(M, K, O, G, fixed_point)
    if ws is None and nb:
        ws = torch.empty(nb, dtype=torch.uint8, device=device)
    return ws, nb


def fgq_gemm_ws(q, bits, sx, M, K, codes, alpha, O, G, prepared=None, out_bits=0, out_scale=None, out=None,
                ws=None):
    """fgq_gemm / fgq_gemm_q with K split over workgroups when that helps."""
    out = _dfp_out((M,), O, out_bits, q.device, out)
    ws, nb = _ws_for(M, K, O, G, False, q.device, ws)
    rc = lib().fgq_gemm_ws(_dev(q, torch.uint8, "q"), bits, _dev(sx, torch.float32, "sx"), M, K,
                           _dev(codes, torch.uint8, "codes"), _dev(alpha, torch.float32, "alpha"),
                           None if prepared is None else _dev(prepared, torch.uint8, "prepared"), O, G, out_bits,
                           None if out_scale is None else _dev(out_scale, torch.float32, "out_scale"),
                           ctypes.c_void_p(out.data_ptr()),
                           None if ws is None else ctypes.c_void_p(ws.data_ptr()),
                           ws.numel() if ws is not None else 0, _stream())
    _check(rc, "fgq_gemm_ws")
    return out


def fgq_conv2d_dfp_residual(q, bits, sx, shape, codes, prepared, O, R, S, stride, pad, G, res, out_bits=0,
                            out_scale=None, y=None, q_out=None):
    """fgq_conv2d_dfp with a residual block's shortcut addition and ReLU
    fused: y = max(layer + res, 0); with out_bits 8 or 4 also the codes of y
    at out_scale.  Returns y, or (y, q_out) when out_bits is not 0."""
    B, H, W, C = shape
    sh, sw = _pair(stride)
    ph, pw = _pair(pad)
    Ho, Wo = conv_out_hw(H, W, R, S, (sh, sw), (ph, pw))
    n = B * Ho * Wo * O
    if y is None:
        y = torch.empty((B, Ho, Wo, O), dtype=torch.float32, device=q.device)
    if out_bits and q_out is None:
        q_out = torch.empty((B, Ho, Wo, O * out_bits // 8), dtype=torch.uint8, device=q.device)
    checks = [(res, "res", n), (y, "y", n)] + ([(q_out, "q_out", n * out_bits // 8)] if out_bits else [])
    for t, name, want in checks:
        if isinstance(t, torch.Tensor) and t.numel() != want:
            raise ValueError(f"{name} must hold {want} values, got {t.numel()}")
    rc = lib().fgq_conv2d_dfp_residual(_dev(q, torch.uint8, "q"), bits, _dev(sx, torch.float32, "sx"), B, H, W, C,
                                       _dev(codes, torch.uint8, "codes"), _dev(prepared, torch.uint8, "prepared"),
                                       O, R, S, sh, sw, ph, pw, G, _dev(res, torch.float32, "res"),
                                       _dev(y, torch.float32, "y"), out_bits,
                                       None if not out_bits else _dev(out_scale, torch.float32, "out_scale"),
                                       None if not out_bits else _dev(q_out, torch.uint8, "q_out"), _stream())
    _check(rc, "fgq_conv2d_dfp_residual")
    return (y, q_out) if out_bits else y


def fgq_gemm_dfp_ws(q, bits, sx, M, K, codes, prepared, O, G, out_bits=0, out_scale=None, out=None, ws=None):
    """fgq_gemm_dfp with K split over workgroups when that helps."""
    out = _dfp_out((M,), O, out_bits, q.device, out)
    ws, nb = _ws_for(M, K, O, G, True, q.device, ws)
    rc = lib().fgq_gemm_dfp_ws(_dev(q, torch.uint8, "q"), bits, _dev(sx, torch.float32, "sx"), M, K,
                               _dev(codes, torch.uint8, "codes"), _dev(prepared, torch.uint8, "prepared"), O, G,
                               out_bits, None if out_scale is None else _dev(out_scale, torch.float32, "out_scale"),
                               ctypes.c_void_p(out.data_ptr()),
                               None if ws is None else ctypes.c_void_p(ws.data_ptr()),
                               ws.numel() if ws is not None else 0, _stream())
    _check(rc, "fgq_gemm_dfp_ws")
    return out


def fgq_prepare_weights_w8(w, prepared=None):
    """First layer at 8-bit weights: w fp32 [O][C][R][S] -> opaque uint8 buffer."""
    O, C, R, S = w.shape
    nb = int(lib().fgq_prepared_bytes_w8(O, C, R, S))
    if prepared is None:
        prepared = torch.empty(nb, dtype=torch.uint8, device=w.device)
    if prepared.data_ptr() % 256:
        raise ValueError("prepared buffer must be 256-byte aligned")
    rc = lib().fgq_prepare_weights_w8(_dev(w, torch.float32, "w"), O, C, R, S,
                                      ctypes.c_void_p(prepared.data_ptr()), nb, _stream())
    _check(rc, "fgq_prepare_weights_w8")
    return prepared


def fgq_conv2d_w8(q, bits, sx, shape, prepared, O, R, S, stride, pad, out_bits=0, out_scale=None, out=None):
    B, H, W, C = shape
    sh, sw = _pair(stride)
    ph, pw = _pair(pad)
    Ho, Wo = conv_out_hw(H, W, R, S, (sh, sw), (ph, pw))
    out = _dfp_out((B, Ho, Wo), O, out_bits, q.device, out)
    rc = lib().fgq_conv2d_w8(_dev(q, torch.uint8, "q"), bits, _dev(sx, torch.float32, "sx"), B, H, W, C,
                             _dev(prepared, torch.uint8, "prepared"), O, R, S, sh, sw, ph, pw, out_bits,
                             None if out_scale is None else _dev(out_scale, torch.float32, "out_scale"),
                             ctypes.c_void_p(out.data_ptr()), _stream())
    _check(rc, "fgq_conv2d_w8")
    return out


def fgq_group_sums(q, bits, shape, codes, O, R, S, stride, pad, G, row0, nrows, P=None):
    B, H, W, C = shape
    sh, sw = _pair(stride)
    ph, pw = _pair(pad)
    K = R * S * C
    if P is None:
        P = torch.empty((nrows, O, K // G), dtype=torch.int32, device=q.device)
    rc = lib().fgq_group_sums(_dev(q, torch.uint8, "q"), bits, B, H, W, C, _dev(codes, torch.uint8, "codes"),
                              O, R, S, sh, sw, ph, pw, G, row0, nrows, _dev(P, torch.int32, "P"), _stream())
    _check(rc, "fgq_group_sums")
    return P


def fgq_probe_mfma_i8(blocks, iters, out=None):
    """Measurement utility: blocks * iters * 16 * 65536 int8 matrix operations
    (see include/fgq.h); returns the int32 sink [blocks * 256]."""
    if out is None:
        out = torch.empty(blocks * 256, dtype=torch.int32, device="cuda")
    rc = lib().fgq_probe_mfma_i8(blocks, iters, _dev(out, torch.int32, "out"), out.numel(), _stream())
    _check(rc, "fgq_probe_mfma_i8")
    return out
