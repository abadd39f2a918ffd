"""Calls on distinct streams from several host threads (the boundary's
thread-safety convention): four threads, each with its own stream and
buffers, run quantization, the folded (G=4) and per-group (G=64)
convolutions and a GEMM many times over while the others do the same; every
result must equal the one computed by a single thread beforehand, bit for
bit.  The binding releases the interpreter lock inside each library call,
so the library's host code runs concurrently.
"""
import threading

import numpy as np
import pytest
import torch

import fgq_inputs as fi

fgq = pytest.importorskip("paper_1705_01462_amd")

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]


def test_threads_on_distinct_streams_match_serial():
    B, H, W, C, O, R, S = 2, 12, 12, 128, 96, 3, 3
    K = R * S * C
    layers = {}
    for G in (4, 64):
        w = fi.he_weights(O, C, R, S, "threads", G)
        codes, alpha, _ = fgq.fgq_ternarize(torch.from_numpy(w).cuda(), G)
        layers[G] = (codes, alpha, fgq.fgq_prepare_weights(codes, alpha, O, K, G))
    MG, KG, OG = 24, 512, 80
    wg = fi.gauss_weights(OG, KG, 0.05, "threads-gemm")
    cg, ag, _ = fgq.fgq_ternarize(torch.from_numpy(wg).cuda(), 4)
    pg = fgq.fgq_prepare_weights(cg, ag, OG, KG, 4)
    nthreads, reps = 4, 20

    def make(t):
        x = torch.from_numpy(fi.relu_gauss((B, H, W, C), "threads-x", t)).cuda()
        xg = torch.from_numpy(fi.relu_gauss((MG, KG), "threads-xg", t)).cuda()
        n = x.numel()
        return dict(x=x, xg=xg, q=torch.empty(n, dtype=torch.uint8, device="cuda"),
                    sx=torch.empty(1, device="cuda"),
                    ws=torch.empty(fgq.fgq_quantize_ws_bytes(n), dtype=torch.uint8, device="cuda"),
                    qg=torch.empty(xg.numel(), dtype=torch.uint8, device="cuda"),
                    sxg=torch.empty(1, device="cuda"),
                    wsg=torch.empty(fgq.fgq_quantize_ws_bytes(xg.numel()), dtype=torch.uint8, device="cuda"),
                    y4=torch.empty((B, H, W, O), device="cuda"), y64=torch.empty((B, H, W, O), device="cuda"),
                    yg=torch.empty((MG, OG), device="cuda"))

    def run(b):
        fgq.fgq_quantize_act(b["x"], 8, q=b["q"], scale_out=b["sx"], ws=b["ws"])
        for G in (4, 64):
            codes, alpha, prep = layers[G]
            fgq.fgq_conv2d(b["q"], 8, b["sx"], (B, H, W, C), codes, alpha, O, R, S, 1, 1, G, prepared=prep,
                           y=b[f"y{G}"])
        fgq.fgq_quantize_act(b["xg"], 8, q=b["qg"], scale_out=b["sxg"], ws=b["wsg"])
        fgq.fgq_gemm(b["qg"], 8, b["sxg"], MG, KG, cg, ag, OG, 4, prepared=pg, y=b["yg"])

    keys = ("q", "sx", "y4", "y64", "qg", "sxg", "yg")
    bufs = [make(t) for t in range(nthreads)]
    for b in bufs:
        run(b)
    torch.cuda.synchronize()
    serial = [{k: b[k].clone() for k in keys} for b in bufs]
    errors = []
    start = threading.Barrier(nthreads)

    def worker(t):
        try:
            s = torch.cuda.Stream()
            b = bufs[t]
            start.wait()
            with torch.cuda.stream(s):
                for rep in range(reps):
                    for k in keys:
                        b[k].zero_()
                    run(b)
                    s.synchronize()
                    for k in keys:
                        if not torch.equal(b[k], serial[t][k]):
                            errors.append(f"thread {t} repetition {rep}: {k} differs from the serial result")
                            return
        except Exception as e:  # reported by the main thread
            errors.append(f"thread {t}: {e!r}")

    threads = [threading.Thread(target=worker, args=(t,)) for t in range(nthreads)]
    for th in threads:
        th.start()
    for th in threads:
        th.join(timeout=120)
    assert not any(th.is_alive() for th in threads), "a worker thread did not finish"
    assert not errors, errors[:4]
    # the threads' inputs differ, so agreement is not vacuous
    assert not np.array_equal(serial[0]["y4"].cpu().numpy(), serial[1]["y4"].cpu().numpy())
