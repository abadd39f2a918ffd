"""GPU parity: the HIP path (through the C ABI) against the CPU oracle on the
same seeded inputs.

Bars: ternary codes, alpha, Delta, quantized activations,
the scale and int32 group sums are bit-exact; the direct per-group layer
kernel (fp64 alpha epilogue) is bit-exact too; the matrix-core kernels
(folded-scale for G != 64, per-group for G = 64) are within 1e-5 of the
summand magnitude s_x * sum_g alpha_g |P_g| element-wise and within 1e-5
normwise.
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


def sampled_rows(M, seed, tile=64, ntiles=64):
    """4096 rows of an M-row layer (all of them if fewer): whole tiles, the
    first and last, the first and last of each eighth of the range, the rest
    seeded and scattered."""
    nt = (M + tile - 1) // tile
    if nt <= ntiles:
        return np.arange(M)
    must = {0, nt - 1}
    for x in range(8):
        must.add(x * nt // 8)
        must.add((x + 1) * nt // 8 - 1)
    rest = np.setdiff1d(np.arange(nt), sorted(must))
    pick = np.random.default_rng(seed).choice(rest, ntiles - len(must), replace=False)
    tiles = np.sort(np.concatenate([sorted(must), pick]))
    rows = (tiles[:, None] * tile + np.arange(tile)[None, :]).ravel()
    return rows[rows < M]


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def ref_layer(w, x, G, bits, R, S, stride, pad, rows=None):
    """Oracle pipeline: ternarize, pack, quantize, conv (optionally a row range)."""
    O = w.shape[0]
    t, a, d = oracle.ternarize(w, G)
    codes = oracle.pack_codes(t)
    q, s = oracle.quantize_act(x, bits)
    y = oracle.conv2d(q, bits, s, x.shape, codes, a, O, R, S, (stride, stride), (pad, pad), G,
                      rows=rows)
    return dict(t=t, a=a, d=d, codes=codes, q=q, s=s, y=y)


def gpu_inputs(w, x, G, bits):
    codes, alpha, delta = fgq.fgq_ternarize(dev(w), G)
    q, sx = fgq.fgq_quantize_act(dev(x), bits)
    return codes, alpha, delta, q, sx


def summand_magnitude(ref, x_shape, G, bits, O, R, S, stride, pad, row0, nrows):
    P = oracle.group_sums_conv(ref["q"], bits, x_shape, ref["codes"], O, R, S, (stride, stride),
                               (pad, pad), G, row0, nrows).astype(np.float64)
    return float(ref["s"]) * np.einsum("mog,og->mo", np.abs(P), ref["a"].astype(np.float64))


def assert_fold_close(y, y_ref, mag):
    """Element-wise within 1e-5 of the summand magnitude, normwise within
    1e-5; also reports the largest relative error over the outputs that are
    not near zero (|y_ref| >= 1e-3 rms)."""
    yr = y_ref.astype(np.float64)
    err = np.abs(y.astype(np.float64) - yr)
    bound = TOL * mag
    bad = err > bound
    assert not bad.any(), f"{bad.sum()} outputs beyond 1e-5 of the summand magnitude; " \
                          f"worst ratio {np.max(err / np.maximum(mag, 1e-300)):.3e}"
    assert np.linalg.norm(err) <= TOL * np.linalg.norm(yr) + 1e-30
    big = np.abs(yr) >= 1e-3 * np.sqrt(np.mean(yr * yr))
    if big.any():
        print(f"[parity] max rel error over |y| >= 1e-3 rms: {np.max(err[big] / np.abs(yr[big])):.2e}; "
              f"max error / summand magnitude: {np.max(err / np.maximum(mag, 1e-300)):.2e}")


# ---------------------------------------------------------------------------
# ternarize / quantize
# ---------------------------------------------------------------------------

TERN_CASES = [
    # O, C, R, S, G, dist
    (16, 64, 3, 3, 4, "he"), (16, 64, 3, 3, 64, "he"), (16, 64, 3, 3, 1, "he"),
    (16, 64, 3, 3, 2, "ties"), (16, 64, 3, 3, 8, "laplace"), (8, 12, 1, 1, 3, "he"),
    (8, 12, 1, 1, 6, "ties"), (5, 256, 1, 1, 128, "laplace"), (1000, 2048, 1, 1, 4, "he"),
    (64, 16, 3, 3, 16, "zeros"), (7, 4, 7, 7, 4, "he"),
    (8, 6, 3, 3, 3, "he"), (5, 10, 1, 1, 5, "ties"),   # K % 4 != 0: rows end mid-byte
]


def make_weights(O, C, R, S, dist, tag):
    if dist == "he":
        return fi.he_weights(O, C, R, S, tag)
    if dist == "laplace":
        return fi.laplace_weights(O, C * R * S, 0.05, tag).reshape(O, C, R, S)
    r = fi.rng("tern", dist, tag)
    if dist == "ties":
        return (r.integers(-3, 4, (O, C, R, S)) * 0.25).astype(np.float32)
    w = fi.he_weights(O, C, R, S, tag)
    w[r.random(w.shape) < 0.5] = 0.0  # "zeros": half exact zeros, some all-zero groups
    return w


@pytest.mark.parametrize("method", [oracle.EXACT, oracle.EXP_LEMMA])
@pytest.mark.parametrize("case", TERN_CASES)
def test_ternarize_bit_exact(case, method):
    O, C, R, S, G, dist = case
    w = make_weights(O, C, R, S, dist, case)
    t, a, d = oracle.ternarize(w, G, method)
    codes, alpha, delta = fgq.fgq_ternarize(dev(w), G, method)
    np.testing.assert_array_equal(host(codes), oracle.pack_codes(t))
    np.testing.assert_array_equal(host(alpha).view(np.uint32), a.view(np.uint32))
    np.testing.assert_array_equal(host(delta).view(np.uint32), d.view(np.uint32))


def test_ternarize_reports_nonfinite():
    w = fi.he_weights(4, 8, 3, 3, "nan")
    w[2, 5, 1, 1] = np.nan
    with pytest.raises(fgq.FgqError) as e:
        fgq.fgq_ternarize(dev(w), 4)
    assert e.value.code == 5
    w[2, 5, 1, 1] = np.inf
    with pytest.raises(fgq.FgqError):
        fgq.fgq_ternarize(dev(w), 4)



def test_ternarize_code_bytes_golden():
    """fgq_ternarize writes the hand-worked bytes of tests/golden/code_bytes.txt
    (the byte layout of include/fgq.h): with groups of one weight, w = t gives
    alpha = |w| and codes t, so the stored bytes are exactly the golden ones."""
    import os
    path = os.path.join(os.path.dirname(__file__), "golden", "code_bytes.txt")
    n = 0
    for line in open(path):
        if line.startswith("#") or not line.strip():
            continue
        K, ts, bs = (p.strip() for p in line.split("|"))
        t = np.array([[int(v) for v in r.split()] for r in ts.split(";")], np.float32)
        b = np.array([[int(v, 16) for v in r.split()] for r in bs.split(";")], np.uint8)
        codes, alpha, _ = fgq.fgq_ternarize(dev(t), 1)
        assert np.array_equal(host(codes), b), f"K={K} t={ts}"
        assert np.array_equal(host(alpha), np.abs(t))
        n += 1
    assert n >= 10

@pytest.mark.parametrize("bits", [8, 4])
@pytest.mark.parametrize("n", [2, 4096 * 16 + 2, 3 * 7 * 5 * 16, 32 * 28 * 28 * 128, 4 * 5_000_003])
@pytest.mark.parametrize("given_scale", [False, True])
def test_quantize_bit_exact(bits, n, given_scale):
    """Odd sizes (tails), the benchmark size and a 20M-value tensor."""
    x = fi.relu_gauss((n,), "quant", bits)
    x[::97] *= -1.0           # some negative inputs
    if n > 100:
        x[7] = np.nan
    scale = np.float32(0.0173) if given_scale else None
    q_ref, s_ref = oracle.quantize_act(x, bits, scale)
    sc = dev(np.array([scale], np.float32)) if given_scale else None
    q, s = fgq.fgq_quantize_act(dev(x), bits, scale_in=sc)
    assert host(s)[0] == s_ref
    np.testing.assert_array_equal(host(q), q_ref)


@pytest.mark.parametrize("bits", [8, 4])
@pytest.mark.parametrize("scale", [0.5, 1.0 / 3.0, 0.0173, 7.0e-30, 3.0e38, 1.0e-39])
def test_quantize_rounding_ties_and_extremes(bits, scale):
    """Quotients at and next to half-integers (round half to even), values
    far beyond the range, +-inf, NaN, zeros and subnormal inputs, for
    scales whose reciprocal is normal (the reciprocal-and-correction path)
    and for a subnormal scale and one with a subnormal reciprocal (the
    ordinary division path)."""
    s32 = np.float32(scale)
    qmax = 255 if bits == 8 else 15
    k = np.arange(0, qmax + 2, dtype=np.float32)
    with np.errstate(over="ignore"):  # the 3e38 scale overflows to inf on purpose
        ties = (k + np.float32(0.5)) * s32                  # float32 products: at or next to ties
        near = np.concatenate([np.nextafter(ties, np.float32(np.inf)), np.nextafter(ties, np.float32(0))])
        r = fi.rng("quant-ties", bits, scale)
        rand = (r.random(4000).astype(np.float32) * np.float32(qmax + 3)) * s32
        special = np.array([0.0, -0.0, np.inf, -np.inf, np.nan, 1e-45, -1e-45, 1e-40, 3.4e38, -3.4e38,
                            s32 * np.float32(1e6), s32], np.float32)
    x = np.concatenate([ties, near, rand, special]).astype(np.float32)
    if x.size % 2:
        x = np.append(x, np.float32(1.0))
    q_ref, s_ref = oracle.quantize_act(x, bits, s32)
    q, sq = fgq.fgq_quantize_act(dev(x), bits, scale_in=dev(np.array([s32], np.float32)))
    assert host(sq)[0] == s_ref
    np.testing.assert_array_equal(host(q), q_ref)


def test_quantize_unaligned_views():
    """Pointers that are not 16-byte aligned take the scalar path."""
    x = fi.relu_gauss((1003 * 2,), "unal")
    xd = dev(x)[1:]
    q_ref, s_ref = oracle.quantize_act(x[1:], 8)
    qbuf = torch.empty(x.size + 16, dtype=torch.uint8, device="cuda")
    q, s = fgq.fgq_quantize_act(xd, 8, q=qbuf[3:3 + xd.numel()])
    assert host(s)[0] == s_ref
    np.testing.assert_array_equal(host(q), q_ref)


# ---------------------------------------------------------------------------
# group sums and layers
# ---------------------------------------------------------------------------

LAYER_CASES = [
    # B, H, W, C, O, R, S, stride, pad, G, bits
    (2, 9, 7, 16, 24, 3, 3, 1, 1, 4, 8),       # K = 144: partial K step, ragged M
    (2, 9, 7, 16, 24, 3, 3, 2, 1, 4, 8),
    (3, 8, 8, 64, 100, 3, 3, 1, 1, 64, 8),     # O not a multiple of the channel tile
    (3, 8, 8, 64, 100, 3, 3, 1, 1, 64, 4),
    (2, 12, 12, 32, 64, 1, 1, 2, 0, 8, 4),
    (1, 5, 5, 128, 130, 3, 3, 1, 1, 4, 8),
    (2, 15, 15, 4, 16, 7, 7, 2, 3, 4, 8),      # conv1-like, C padded to 4
    (2, 15, 15, 4, 40, 7, 7, 2, 3, 4, 4),      # the same with 4-bit activations
    (2, 11, 13, 8, 36, 3, 3, 1, 1, 8, 8),      # C = 8: two taps per 16-channel piece
    (2, 11, 13, 8, 36, 5, 5, 2, 2, 4, 4),
    (2, 6, 6, 6, 5, 3, 3, 1, 1, 3, 8),         # G = 3, C % 4 != 0
    (2, 6, 6, 16, 9, 3, 3, 1, 1, 1, 4),        # G = 1
    (4, 14, 14, 256, 64, 1, 1, 1, 0, 64, 8),
    # input-patch staging (C % 128 == 0, R*S > 1, O > 64): several chunks,
    # 4-bit activations, stride 2, a 5x5 filter, tiles spanning images, and
    # G = 64 beyond 160 groups (folded layout)
    (2, 9, 11, 256, 72, 3, 3, 1, 1, 4, 4),
    (3, 12, 10, 384, 130, 3, 3, 2, 1, 4, 8),
    (2, 8, 8, 128, 96, 5, 5, 1, 2, 4, 8),
    (5, 5, 5, 256, 128, 3, 3, 1, 1, 4, 8),
    (1, 6, 6, 1280, 80, 3, 3, 1, 1, 64, 8),
]


@pytest.mark.parametrize("case", LAYER_CASES)
def test_group_sums_bit_exact(case):
    B, H, W, C, O, R, S, st, pd, G, bits = case
    w = fi.he_weights(O, C, R, S, "gs", case)
    x = fi.relu_gauss((B, H, W, C), "gs", case)
    t, a, _ = oracle.ternarize(w, G)
    q_ref, _ = oracle.quantize_act(x, bits)
    codes, alpha, _, q, sx = gpu_inputs(w, x, G, bits)
    Ho, Wo = fi.conv_out(H, W, R, S, st, pd)
    M = B * Ho * Wo
    for row0, nrows in [(0, min(M, 70)), (M - min(M, 33), min(M, 33))]:
        P_ref = oracle.group_sums_conv(q_ref, bits, (B, H, W, C), oracle.pack_codes(t), O, R, S,
                                       (st, st), (pd, pd), G, row0, nrows)
        P = fgq.fgq_group_sums(q, bits, (B, H, W, C), codes, O, R, S, st, pd, G, row0, nrows)
        np.testing.assert_array_equal(host(P), P_ref)


@pytest.mark.parametrize("case", LAYER_CASES)
def test_conv_direct_path_bit_exact(case):
    B, H, W, C, O, R, S, st, pd, G, bits = case
    w = fi.he_weights(O, C, R, S, "direct", case)
    x = fi.relu_gauss((B, H, W, C), "direct", case)
    ref = ref_layer(w, x, G, bits, R, S, st, pd)
    codes, alpha, _, q, sx = gpu_inputs(w, x, G, bits)
    y = fgq.fgq_conv2d(q, bits, sx, (B, H, W, C), codes, alpha, O, R, S, st, pd, G)
    yh = host(y).reshape(-1, O)
    np.testing.assert_array_equal(yh.view(np.uint32), ref["y"].view(np.uint32))


@pytest.mark.parametrize("case", LAYER_CASES)
def test_conv_folded_path(case):
    B, H, W, C, O, R, S, st, pd, G, bits = case
    w = fi.he_weights(O, C, R, S, "fold", case)
    if G < 4:
        # with one or two weights per group the scales of random weights come
        # arbitrarily close to zero, which the folded layout's accuracy guard
        # rejects (test_gpu_guard.py); here magnitudes are kept >= sigma / 4
        sd = np.float32(np.sqrt(2.0 / (C * R * S)))
        w = np.where(w < 0, -1.0, 1.0).astype(np.float32) * np.maximum(np.abs(w), sd / 4)
    x = fi.relu_gauss((B, H, W, C), "fold", case)
    ref = ref_layer(w, x, G, bits, R, S, st, pd)
    codes, alpha, _, q, sx = gpu_inputs(w, x, G, bits)
    K = R * S * C
    prep = fgq.fgq_prepare_weights(codes, alpha, O, K, G)
    y = fgq.fgq_conv2d(q, bits, sx, (B, H, W, C), codes, alpha, O, R, S, st, pd, G, prepared=prep)
    yh = host(y).reshape(-1, O)
    mag = summand_magnitude(ref, x.shape, G, bits, O, R, S, st, pd, 0, yh.shape[0])
    assert_fold_close(yh, ref["y"], mag)
    # deterministic: a second launch gives identical bits
    y2 = fgq.fgq_conv2d(q, bits, sx, (B, H, W, C), codes, alpha, O, R, S, st, pd, G, prepared=prep)
    np.testing.assert_array_equal(host(y2), host(y))


@pytest.mark.parametrize("bits", [8, 4])
@pytest.mark.parametrize("folded", [False, True])
def test_gemm_single_layer(bits, folded):
    """Single FGQ GEMM: M=64, K=256, O=128, W ~ N(0, 0.05^2), G=4."""
    M, K, O, G = 64, 256, 128, 4
    w = fi.gauss_weights(O, K, 0.05, "gemm1")
    x = fi.relu_gauss((M, K), "gemm1")
    t, a, _ = oracle.ternarize(w, G)
    codes_ref = oracle.pack_codes(t)
    q_ref, s_ref = oracle.quantize_act(x, bits)
    y_ref = oracle.gemm(q_ref, bits, s_ref, M, K, codes_ref, a, O, G)
    codes, alpha, _ = fgq.fgq_ternarize(dev(w), G)
    q, sx = fgq.fgq_quantize_act(dev(x), bits)
    prep = fgq.fgq_prepare_weights(codes, alpha, O, K, G) if folded else None
    y = host(fgq.fgq_gemm(q, bits, sx, M, K, codes, alpha, O, G, prepared=prep))
    if folded:
        P = oracle.group_sums_conv(q_ref, bits, (1, M, 1, K), codes_ref, O, 1, 1, (1, 1), (0, 0), G)
        mag = float(s_ref) * np.einsum("mog,og->mo", np.abs(P.astype(np.float64)), a.astype(np.float64))
        assert_fold_close(y, y_ref, mag)
    else:
        np.testing.assert_array_equal(y.view(np.uint32), y_ref.view(np.uint32))


@pytest.mark.parametrize("bits", [8, 4])
@pytest.mark.parametrize("M,K,O", [(64, 256, 128), (77, 640, 40), (40, 64 * 161, 40), (300, 1280, 96),
                                   (70, 1344, 33)])
def test_gemm_group64(bits, M, K, O):
    """G=64 GEMMs with prepared weights: the per-group kernels (K/64 <= 160
    groups, incl. odd group counts, ragged M and O, the largest reduction
    of the persistent kernel (1280) and the next one up) and the
    folded-scale kernel beyond 160 groups."""
    G = 64
    w = fi.gauss_weights(O, K, 0.05, "gemm64", M, K)
    x = fi.relu_gauss((M, K), "gemm64", M, K)
    t, a, _ = oracle.ternarize(w, G)
    codes_ref = oracle.pack_codes(t)
    q_ref, s_ref = oracle.quantize_act(x, bits)
    y_ref = oracle.gemm(q_ref, bits, s_ref, M, K, codes_ref, a, O, G)
    codes, alpha, _ = fgq.fgq_ternarize(dev(w), G)
    q, sx = fgq.fgq_quantize_act(dev(x), bits)
    prep = fgq.fgq_prepare_weights(codes, alpha, O, K, G)
    y = host(fgq.fgq_gemm(q, bits, sx, M, K, codes, alpha, O, G, prepared=prep))
    P = oracle.group_sums_conv(q_ref, bits, (1, M, 1, K), codes_ref, O, 1, 1, (1, 1), (0, 0), G)
    mag = float(s_ref) * np.einsum("mog,og->mo", np.abs(P.astype(np.float64)), a.astype(np.float64))
    assert_fold_close(y, y_ref, mag)


FULL = [
    # conv3_x 3x3 128->128 on 28x28, batch 32, G=4 and G=64; 1x1 256->64 on 56x56, G=64
    (32, 28, 28, 128, 128, 3, 3, 1, 1, 4, 8),
    (32, 28, 28, 128, 128, 3, 3, 1, 1, 64, 8),
    (32, 56, 56, 256, 64, 1, 1, 1, 0, 64, 8),
]


@pytest.mark.parametrize("case", FULL)
def test_full_size_layers_sampled_rows(case):
    """Full-size layers, launched exactly as the benchmark launches them;
    the oracle computes 4096 sampled rows (64 tiles of 64, scattered, the
    first and last tile and those at each eighth of the range included)."""
    B, H, W, C, O, R, S, st, pd, G, bits = case
    w = fi.he_weights(O, C, R, S, "full", case)
    x = fi.relu_gauss((B, H, W, C), "full", case)
    codes, alpha, _, q, sx = gpu_inputs(w, x, G, bits)
    t, a, _ = oracle.ternarize(w, G)
    codes_ref = oracle.pack_codes(t)
    q_ref, s_ref = oracle.quantize_act(x, bits)
    np.testing.assert_array_equal(host(codes), codes_ref)
    np.testing.assert_array_equal(host(q), q_ref)
    K = R * S * C
    prep = fgq.fgq_prepare_weights(codes, alpha, O, K, G)
    y_fold = host(fgq.fgq_conv2d(q, bits, sx, (B, H, W, C), codes, alpha, O, R, S, st, pd, G,
                                 prepared=prep)).reshape(-1, O)
    y_dir = host(fgq.fgq_conv2d(q, bits, sx, (B, H, W, C), codes, alpha, O, R, S, st, pd, G)).reshape(-1, O)
    M = y_fold.shape[0]
    rows = sampled_rows(M, seed=sum(case))
    y_ref, mag = oracle.conv2d_rows(q_ref, bits, s_ref, x.shape, codes_ref, a, O, R, S, (st, st), (pd, pd), G,
                                    rows)
    assert_fold_close(y_fold[rows], y_ref, mag)
    np.testing.assert_array_equal(y_dir[rows].view(np.uint32), y_ref.view(np.uint32))


@pytest.mark.parametrize("G", [4, 64])
@pytest.mark.parametrize("bits", [8, 4])
def test_degenerate_activations(bits, G):
    """All-zero activations give exactly 0; all-qmax activations give
    s_x * qmax * sum_g alpha_g T_g on both paths."""
    B, H, W, O, R, S = 2, 6, 6, 48, 3, 3
    C = 32 if G == 4 else 64
    w = fi.he_weights(O, C, R, S, "degen")
    codes, alpha, _ = fgq.fgq_ternarize(dev(w), G)
    K = R * S * C
    prep = fgq.fgq_prepare_weights(codes, alpha, O, K, G)
    qmax = 255 if bits == 8 else 15
    nbytes = B * H * W * C if bits == 8 else B * H * W * C // 2
    codes_h, alpha_h = host(codes), host(alpha)
    for val in (0, 255):
        q = torch.full((nbytes,), val, dtype=torch.uint8, device="cuda")
        sx = torch.ones(1, dtype=torch.float32, device="cuda")
        qh = host(q)
        y_ref = oracle.conv2d(qh, bits, 1.0, (B, H, W, C), codes_h, alpha_h, O, R, S, (1, 1), (0, 0), G)
        ref = dict(q=qh, s=np.float32(1.0), codes=codes_h, a=alpha_h)
        mag = summand_magnitude(ref, (B, H, W, C), G, bits, O, R, S, 1, 0, 0, y_ref.shape[0])
        for prep_arg in (None, prep):
            y = host(fgq.fgq_conv2d(q, bits, sx, (B, H, W, C), codes, alpha, O, R, S, 1, 0, G,
                                    prepared=prep_arg)).reshape(-1, O)
            if val == 0:
                assert not y.any()
            elif prep_arg is None:
                np.testing.assert_array_equal(y, y_ref)
            else:
                assert_fold_close(y, y_ref, mag)

