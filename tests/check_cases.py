"""A spread of layer calls over every kernel family, for two GPU checks
(tests/test_gpu_check.py):

* the checking build (libfgq_check.so, loaded with FGQ_LIBRARY=check in a
  child process) runs them and must report no out-of-bounds access and
  produce the same bytes as the normal library;
* the normal library runs them twice in one process and must produce the
  same bytes both times (a data race through LDS or between workgroups would
  show as run-to-run differences).

Shapes are ragged on purpose (rows, channels and K not multiples of the
tiles, K not a multiple of the 128-wide step, strides, 1x1 and 3x3, C = 4)
and include seeded random layer shapes.  Run as a script with an output
folder to save every result as .npy (the child process of the check).
"""
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import fgq_inputs as fi  # noqa: E402

# B H W C O R S stride pad G bits
CONV = [
    (2, 9, 11, 64, 72, 3, 3, 1, 1, 4, 8),
    (1, 13, 7, 128, 96, 3, 3, 2, 1, 64, 8),
    (2, 6, 6, 192, 40, 1, 1, 1, 0, 64, 4),
    (1, 10, 10, 96, 130, 3, 3, 1, 1, 3, 8),
    (2, 12, 12, 4, 64, 7, 7, 2, 3, 4, 8),
    (3, 8, 8, 64, 256, 1, 1, 1, 0, 4, 8),
    (1, 5, 5, 64 * 162 // 9, 33, 3, 3, 1, 1, 64, 4),
]
# M K O G bits
GEMM = [(64, 1152, 200, 4, 8), (1, 4096, 96, 4, 8), (37, 640, 40, 64, 4), (9, 384, 70, 8, 8)]


def random_convs(n=4):
    """Seeded random layer shapes within modest bounds."""
    r = fi.rng("check-cases-shapes")
    out = []
    for _ in range(n):
        G = int(r.choice([4, 64]))
        C = int(r.choice([64, 128, 192])) if G == 64 else int(r.integers(2, 40)) * 4
        R = int(r.choice([1, 3]))
        out.append((int(r.integers(1, 4)), int(r.integers(4, 17)), int(r.integers(4, 17)), C,
                    int(r.integers(1, 200)), R, R, int(r.choice([1, 2])), R // 2, G, int(r.choice([8, 4]))))
    return out


def run_cases(fgq, torch):
    """Every call's output as a host numpy array, by name."""
    def dev(a):
        return torch.from_numpy(np.ascontiguousarray(a)).cuda()

    def host(t):
        torch.cuda.synchronize()
        return t.cpu().numpy()

    res = {}
    for i, case in enumerate(CONV + random_convs()):
        B, H, W, C, O, R, S, st, pd, G, bits = case
        tag = f"conv{i}"
        w = fi.he_weights(O, C, R, S, "check", *case)
        x = fi.relu_gauss((B, H, W, C), "check", *case)
        codes, alpha, delta = fgq.fgq_ternarize(dev(w), G)
        res[tag + "_codes"], res[tag + "_alpha"] = host(codes), host(alpha)
        q, sx = fgq.fgq_quantize_act(dev(x), bits)
        res[tag + "_q"] = host(q)
        K = R * S * C
        prep = fgq.fgq_prepare_weights(codes, alpha, O, K, G, fallback=True)
        shape = (B, H, W, C)
        y = fgq.fgq_conv2d(q, bits, sx, shape, codes, alpha, O, R, S, st, pd, G, prepared=prep)
        res[tag + "_y"] = host(y)
        res[tag + "_ydirect"] = host(fgq.fgq_conv2d(q, bits, sx, shape, codes, alpha, O, R, S, st, pd, G))
        shortcut = dev(fi.rng("check-res", *case).standard_normal(res[tag + "_y"].shape).astype(np.float32))
        res[tag + "_res"] = host(fgq.fgq_conv2d_residual(q, bits, sx, shape, codes, alpha, O, R, S, st, pd, G,
                                                         shortcut, prepared=prep))
        res[tag + "_resdirect"] = host(fgq.fgq_conv2d_residual(q, bits, sx, shape, codes, alpha, O, R, S, st, pd,
                                                               G, shortcut))
        rsc = dev(np.array([np.float32(0.8 * max(float(res[tag + "_res"].max()), 1e-3) / 255.0)], np.float32))
        yq, qq = fgq.fgq_conv2d_residual_q(q, bits, sx, shape, codes, alpha, O, R, S, st, pd, G, shortcut, 8, rsc,
                                           prepared=prep)
        res[tag + "_resq8"], res[tag + "_resq8y"] = host(qq), host(yq)
        if O % 2 == 0:
            res[tag + "_resq4d"] = host(fgq.fgq_conv2d_residual_q(q, bits, sx, shape, codes, alpha, O, R, S, st,
                                                                  pd, G, shortcut, 4, rsc)[1])
        yh = res[tag + "_y"]
        for ob in (8, 4):
            if ob == 4 and O % 2:
                continue
            sc = dev(np.array([np.float32(0.9 * max(float(yh.max()), 1e-3) / (2 ** ob - 1))], np.float32))
            res[f"{tag}_q{ob}"] = host(fgq.fgq_conv2d_q(q, bits, sx, shape, codes, alpha, O, R, S, st, pd, G, ob,
                                                        sc, prepared=prep))
        prepd = fgq.fgq_prepare_weights_dfp(codes, alpha, O, K, G, 8)
        res[tag + "_dfp"] = host(fgq.fgq_conv2d_dfp(q, bits, sx, shape, codes, prepd, O, R, S, st, pd, G))
        M = res[tag + "_y"].size // O
        n = min(M, 50)
        res[tag + "_P"] = host(fgq.fgq_group_sums(q, bits, shape, codes, O, R, S, st, pd, G, M - n, n))
    for i, (M, K, O, G, bits) in enumerate(GEMM):
        tag = f"gemm{i}"
        w = fi.gauss_weights(O, K, 0.05, "check", M, K, O, G)
        x = fi.relu_gauss((M, K), "check", M, K, O, G)
        codes, alpha, _ = fgq.fgq_ternarize(dev(w), G)
        q, sx = fgq.fgq_quantize_act(dev(x), bits)
        res[tag + "_qn"] = host(fgq.fgq_quantize_act_noalloc(dev(x), bits)[0])
        prep = fgq.fgq_prepare_weights(codes, alpha, O, K, G, fallback=True)
        res[tag + "_y"] = host(fgq.fgq_gemm(q, bits, sx, M, K, codes, alpha, O, G, prepared=prep))
        res[tag + "_ws"] = host(fgq.fgq_gemm_ws(q, bits, sx, M, K, codes, alpha, O, G, prepared=prep))
        prepd = fgq.fgq_prepare_weights_dfp(codes, alpha, O, K, G, 8)
        res[tag + "_dfp"] = host(fgq.fgq_gemm_dfp(q, bits, sx, M, K, codes, prepd, O, G))
        res[tag + "_dfpws"] = host(fgq.fgq_gemm_dfp_ws(q, bits, sx, M, K, codes, prepd, O, G))
    # the first layer at 8-bit weights, ternarization variants, odd-length quantization
    w = fi.he_weights(24, 4, 7, 7, "check-w8")
    x = fi.relu_gauss((2, 20, 20, 4), "check-w8")
    q, sx = fgq.fgq_quantize_act(dev(x), 8)
    prep = fgq.fgq_prepare_weights_w8(dev(w))
    res["w8_y"] = host(fgq.fgq_conv2d_w8(q, 8, sx, (2, 20, 20, 4), prep, 24, 7, 7, 2, 3))
    wv = fi.laplace_weights(20, 72, 0.05, "check-var")
    for m in (fgq.FGQ_TERN_EXP_LEMMA, fgq.FGQ_TERN_GAUSS, fgq.FGQ_TERN_KS):
        c, a, _ = fgq.fgq_ternarize(dev(wv), 8, method=m)
        res[f"tern{m}_codes"], res[f"tern{m}_alpha"] = host(c), host(a)
    c, a, dp, dn = fgq.fgq_ternarize_asym(dev(wv), 8)
    res["asym_codes"], res["asym_dp"] = host(c), host(dp)
    for n in (1, 4097, 12345):
        xs = fi.relu_gauss((n,), "check-q", n)
        res[f"quant{n}"] = host(fgq.fgq_quantize_act(dev(xs), 8)[0])
    return res


def main(outdir):
    import torch

    import paper_1705_01462_amd as fgq
    print(f"[check_cases] library {os.path.basename(fgq.LIB_PATH)}", flush=True)
    res = run_cases(fgq, torch)
    n, site, off = fgq.fgq_check_violations()
    os.makedirs(outdir, exist_ok=True)
    for k, v in res.items():
        np.save(os.path.join(outdir, k + ".npy"), v)
    print(f"[check_cases] {len(res)} results; violations {n} (first site {site}, offset {off})", flush=True)
    with open(os.path.join(outdir, "violations.txt"), "w") as f:
        f.write(f"{n} {site} {off}\n")


if __name__ == "__main__":
    main(sys.argv[1])
