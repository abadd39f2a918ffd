"""The CPU oracle under AddressSanitizer, UndefinedBehaviorSanitizer and the
leak checker (no GPU).

The oracle's C source is compiled with a small driver
(tests/oracle_check_main.c) into one executable with
-fsanitize=address,undefined and no recovery, so any out-of-bounds access,
use after free, signed overflow, misaligned or invalid shift, or leaked
allocation ends the run with a report.  Every routine runs on small seeded
inputs that reach its edge cases (ragged K, K not a multiple of 4, padding,
strides, 4-bit activations, a supplied and a dynamic scale, zero and
all-maximal data), and its outputs are compared byte for byte with the
regular build of the oracle, so the sanitized build is checked to compute
the same thing.
"""
import os
import shutil
import subprocess

import numpy as np
import pytest

import fgq_inputs as fi
import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "fgq_oracle.c")
DRIVER = os.path.join(ROOT, "tests", "oracle_check_main.c")


@pytest.fixture(scope="module")
def exe(tmp_path_factory):
    if shutil.which("gcc") is None:
        pytest.skip("gcc not available")
    out = str(tmp_path_factory.mktemp("orcsan") / "oracle_check")
    cmd = ["gcc", "-O1", "-g", "-std=c11", "-fno-fast-math", "-ffp-contract=off", "-fopenmp",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer",
           "-Wall", "-Wextra", "-I", os.path.join(ROOT, "oracle"), "-o", out, SRC, DRIVER, "-lm"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0 and "asan" in (r.stderr or "").lower():
        pytest.skip("sanitizer runtime not available: " + r.stderr[-300:])
    assert r.returncode == 0, r.stderr
    return out


def run(exe, args, *arrays):
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0:halt_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1", OMP_NUM_THREADS="2")
    data = b"".join(np.ascontiguousarray(a).tobytes() for a in arrays)
    r = subprocess.run([exe] + [str(x) for x in args], input=data, capture_output=True, env=env,
                       timeout=300)
    assert r.returncode == 0, r.stderr.decode(errors="replace")[-4000:]
    assert b"runtime error" not in r.stderr, r.stderr.decode(errors="replace")[-4000:]
    return r.stdout


def split(buf, *specs):
    """Cut the driver's output into arrays of the given (dtype, count)."""
    out, pos = [], 0
    for dt, n in specs:
        nb = np.dtype(dt).itemsize * n
        out.append(np.frombuffer(buf[pos:pos + nb], dtype=dt))
        pos += nb
    assert pos == len(buf), (pos, len(buf))
    return out


def same(a, b):
    """Byte-for-byte equality of the driver's array a and the regular build's b."""
    assert np.ascontiguousarray(b, dtype=a.dtype).ravel().tobytes() == a.tobytes()


def fsx(s):
    """A float32 scale as an exact decimal argument."""
    return repr(float(np.float32(s)))


TERN_CASES = [(5, 6, 3, 3, 3, 0), (4, 16, 1, 1, 4, 3), (3, 12, 3, 3, 4, 1), (6, 64, 1, 1, 64, 3),
              (2, 5, 1, 3, 5, 4), (4, 9, 2, 2, 1, 0)]


@pytest.mark.parametrize("O,C,R,S,G,method", TERN_CASES)
def test_ternarize(exe, O, C, R, S, G, method):
    w = fi.he_weights(O, C, R, S, "san-tern", O, C, G, method)
    w[0, 0, 0, 0] = 0.0  # a zero weight in the first group
    K = C * R * S
    t, a, d = split(run(exe, ["ternarize", O, C, R, S, G, method], w),
                    (np.int8, O * K), (np.float32, O * K // G), (np.float32, O * K // G))
    t0, a0, d0 = oracle.ternarize(w, G, method)
    same(t, t0), same(a, a0), same(d, d0)


def test_ternarize_asym_and_ks(exe):
    O, C, R, S, G = 3, 8, 3, 3, 8
    w = fi.he_weights(O, C, R, S, "san-asym")
    ng = O * C * R * S // G
    t, a, dp, dn = split(run(exe, ["ternarize_asym", O, C, R, S, G], w),
                         (np.int8, O * C * R * S), (np.float32, ng), (np.float32, ng), (np.float32, ng))
    r = oracle.ternarize_asym(w, G)
    for x, y in zip((t, a, dp, dn), r):
        same(x, y)
    for n in (1, 100, 40000):  # below, near and above the K-S sample size
        x = fi.laplace_weights(1, n, 0.05, "san-ks", n).ravel()
        (d,) = split(run(exe, ["ks", n], x), (np.float64, 2))
        assert tuple(d) == oracle.ks_distances(x)


@pytest.mark.parametrize("O,K", [(1, 1), (3, 5), (2, 8), (4, 13)])
def test_codes(exe, O, K):
    t = fi.rng("san-codes", O, K).integers(-1, 2, (O, K)).astype(np.int8)
    c, t2 = split(run(exe, ["codes", O, K], t), (np.uint8, O * ((K + 3) // 4)), (np.int8, O * K))
    same(c, oracle.pack_codes(t))
    same(t2, t)


@pytest.mark.parametrize("n,bits,scaled", [(1, 8, 0), (7, 8, 0), (1000, 8, 1), (2, 4, 0), (998, 4, 1)])
def test_quantize(exe, n, bits, scaled):
    x = fi.relu_gauss((n,), "san-q", n, bits).astype(np.float32)
    if n > 2:
        x[1] = np.inf
        x[2] = -3.0
    s_in = np.float32(0.0125)
    args = [x] + ([np.array([s_in], np.float32)] if scaled else [])
    nb = n if bits == 8 else n // 2
    q, s = split(run(exe, ["quantize", n, bits, scaled], *args), (np.uint8, nb), (np.float32, 1))
    q0, s0 = oracle.quantize_act(x, bits, s_in if scaled else None)
    same(q, q0)
    assert s[0].tobytes() == np.float32(s0).tobytes()


CONV_CASES = [  # B H W C O R S sh sw ph pw G bits
    (2, 5, 6, 8, 5, 3, 3, 1, 1, 1, 1, 4, 8),
    (1, 7, 5, 6, 3, 3, 3, 2, 2, 1, 1, 3, 8),
    (2, 4, 4, 16, 4, 1, 1, 1, 1, 0, 0, 16, 4),
    (1, 9, 9, 4, 2, 5, 3, 2, 1, 2, 0, 4, 4),
    (1, 3, 3, 2, 2, 3, 3, 1, 1, 1, 1, 1, 8),
]


def conv_inputs(case):
    B, H, W, C, O, R, S, sh, sw, ph, pw, G, bits = case
    w = fi.he_weights(O, C, R, S, "san-conv", *case)
    t, a, _ = oracle.ternarize(w, G)
    codes = oracle.pack_codes(t)
    x = fi.relu_gauss((B, H, W, C), "san-conv-x", *case)
    x.reshape(-1)[:3] = x.max()  # a few maximal codes
    q, sx = oracle.quantize_act(x, bits)
    return q, sx, codes, a


@pytest.mark.parametrize("case", CONV_CASES)
def test_conv_routines(exe, case):
    B, H, W, C, O, R, S, sh, sw, ph, pw, G, bits = case
    geom = [B, H, W, C, O, R, S, sh, sw, ph, pw]
    q, sx, codes, a = conv_inputs(case)
    Ho, Wo = oracle.conv_out_hw(H, W, R, S, (sh, sw), (ph, pw))
    M, K = B * Ho * Wo, R * S * C
    shape, st, pd = (B, H, W, C), (sh, sw), (ph, pw)
    # group sums on a row range that ends at the last row
    row0 = M // 3
    (P,) = split(run(exe, ["group_sums"] + geom + [G, bits, row0, M - row0], q, codes),
                 (np.int32, (M - row0) * O * (K // G)))
    same(P, oracle.group_sums_conv(q, bits, shape, codes, O, R, S, st, pd, G, row0, M - row0))
    (y,) = split(run(exe, ["conv2d"] + geom + [G, bits, fsx(sx), 0, -1], q, codes, a),
                 (np.float32, M * O))
    same(y, oracle.conv2d(q, bits, sx, shape, codes, a, O, R, S, st, pd, G))
    rows = np.array(sorted({0, M - 1, M // 2, 1 % M}), np.int64)
    y, mag = split(run(exe, ["conv2d_rows"] + geom + [G, bits, fsx(sx), len(rows)], q, codes, a, rows),
                   (np.float32, len(rows) * O), (np.float64, len(rows) * O))
    y0, m0 = oracle.conv2d_rows(q, bits, sx, shape, codes, a, O, R, S, st, pd, G, rows)
    same(y, y0), same(mag, m0)
    A, fl = oracle.dfp_alpha(a, 8)
    (A2, fl2) = split(run(exe, ["dfp_alpha", a.size, 8], a), (np.int8, a.size), (np.int32, 1))
    same(A2, A)
    assert int(fl2[0]) == fl
    (y,) = split(run(exe, ["conv2d_dfp"] + geom + [G, bits, fsx(sx), fl, 0, -1], q, codes, A),
                 (np.float32, M * O))
    same(y, oracle.conv2d_dfp(q, bits, sx, shape, codes, A, fl, O, R, S, st, pd, G))


def test_gemm_routines(exe):
    M, K, O, G, bits = 5, 36, 7, 4, 8
    w = fi.gauss_weights(O, K, 0.05, "san-gemm")
    t, a, _ = oracle.ternarize(w, G)
    codes = oracle.pack_codes(t)
    q, sx = oracle.quantize_act(fi.relu_gauss((M, K), "san-gemm-x"), bits)
    (y,) = split(run(exe, ["gemm", M, K, O, G, bits, fsx(sx)], q, codes, a), (np.float32, M * O))
    same(y, oracle.gemm(q, bits, sx, M, K, codes, a, O, G))
    A, fl = oracle.dfp_alpha(a, 4)
    (y,) = split(run(exe, ["gemm_dfp", M, K, O, G, bits, fsx(sx), fl], q, codes, A), (np.float32, M * O))
    same(y, oracle.gemm_dfp(q, bits, sx, M, K, codes, A, fl, O, G))


def test_first_layer_w8(exe):
    B, H, W, C, O, R, S, sh, sw, ph, pw, bits = 1, 9, 7, 3, 4, 3, 3, 2, 2, 1, 1, 8
    w = fi.he_weights(O, C, R, S, "san-w8")
    q, sx = oracle.quantize_act(fi.relu_gauss((B, H, W, C), "san-w8-x"), bits)
    Ho, Wo = oracle.conv_out_hw(H, W, R, S, (sh, sw), (ph, pw))
    M, nw = B * Ho * Wo, O * C * R * S
    W8, fl, y = split(run(exe, ["w8", B, H, W, C, O, R, S, sh, sw, ph, pw, bits, fsx(sx), 0, -1], w, q),
                      (np.int8, nw), (np.int32, 1), (np.float32, M * O))
    W80, fl0 = oracle.w8_quantize(w)
    same(W8, W80)
    assert int(fl[0]) == fl0
    same(y, oracle.conv2d_w8(q, bits, sx, (B, H, W, C), W80, fl0, O, R, S, (sh, sw), (ph, pw)))
