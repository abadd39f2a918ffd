"""The hot path captured in a HIP graph (as the benchmark runs it): every
replay, with eager work and synchronizations in between, must reproduce the
eager results bit for bit.  Covers the dynamic-scale quantization (two
passes), the folded and per-group convolutions, the row-walking folded
kernel (a 1x1 layer with K = 64 over many row tiles), the fused 8-bit
output, the fixed-point convolution, and the split-K GEMMs with their
reduction (none of them may record a memset); and independent batches as
concurrent chains of one graph.
"""
import numpy as np
import pytest
import torch

import fgq_inputs as fi

fgq = pytest.importorskip("paper_1705_01462_amd")

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]


def test_graph_replays_match_eager():
    B, H, W, C, O, R, S = 4, 14, 14, 128, 128, 3, 3
    K = R * S * C
    x = torch.from_numpy(fi.relu_gauss((B, H, W, C), "graph")).cuda()
    outs = {}
    layers = {}
    for G in (4, 64):
        w = fi.he_weights(O, C, R, S, "graph", G)
        codes, alpha, _ = fgq.fgq_ternarize(torch.from_numpy(w).cuda(), G)
        layers[G] = (codes, alpha, fgq.fgq_prepare_weights(codes, alpha, O, K, G),
                     fgq.fgq_prepare_weights_dfp(codes, alpha, O, K, G, 8))
    M, KF, OF, GF = 32, 4096, 512, 4
    wf = fi.gauss_weights(OF, KF, 0.01, "graph-fc")
    cf, af, _ = fgq.fgq_ternarize(torch.from_numpy(wf).cuda(), GF)
    pf = fgq.fgq_prepare_weights(cf, af, OF, KF, GF)
    pfd = fgq.fgq_prepare_weights_dfp(cf, af, OF, KF, GF, 8)
    xf = torch.from_numpy(fi.relu_gauss((M, KF), "graph-fc")).cuda()
    # a 1x1 layer with K = 64 and 1568 row/channel tiles: the row-walking kernel
    BR, HR, CR, OR = 16, 56, 64, 256
    wr = fi.he_weights(OR, CR, 1, 1, "graph-rows", 4)
    cr, ar, _ = fgq.fgq_ternarize(torch.from_numpy(wr).cuda(), 4)
    pr = fgq.fgq_prepare_weights(cr, ar, OR, CR, 4)
    xr = torch.from_numpy(fi.relu_gauss((BR, HR, HR, CR), "graph-rows")).cuda()

    n = x.numel()
    q = torch.empty(n, dtype=torch.uint8, device="cuda")
    sx = torch.empty(1, device="cuda")
    ws = torch.empty(fgq.fgq_quantize_ws_bytes(n), dtype=torch.uint8, device="cuda")
    qf = torch.empty(xf.numel(), dtype=torch.uint8, device="cuda")
    sxf = torch.empty(1, device="cuda")
    wsf = torch.empty(fgq.fgq_quantize_ws_bytes(xf.numel()), dtype=torch.uint8, device="cuda")
    qr = torch.empty(xr.numel(), dtype=torch.uint8, device="cuda")
    sxr = torch.empty(1, device="cuda")
    wsr = torch.empty(fgq.fgq_quantize_ws_bytes(xr.numel()), dtype=torch.uint8, device="cuda")
    osc = torch.full((1,), 0.05, device="cuda")
    Ho = H
    for key in ("y4", "y64", "yd4", "yd64"):
        outs[key] = torch.empty((B, Ho, Ho, O), device="cuda")
    outs["q8"] = torch.empty(B * Ho * Ho * O, dtype=torch.uint8, device="cuda")
    outs["gf"] = torch.empty((M, OF), device="cuda")
    outs["gfd"] = torch.empty((M, OF), device="cuda")
    outs["yr"] = torch.empty((BR, HR, HR, OR), device="cuda")
    outs["qr8"] = torch.empty(BR * HR * HR * OR, dtype=torch.uint8, device="cuda")
    wsg = torch.empty(max(fgq.fgq_gemm_ws_bytes(M, KF, OF, GF, False), 4), dtype=torch.uint8, device="cuda")
    wsgd = torch.empty(max(fgq.fgq_gemm_ws_bytes(M, KF, OF, GF, True), 4), dtype=torch.uint8, device="cuda")

    def step():
        fgq.fgq_quantize_act(x, 8, q=q, scale_out=sx, ws=ws)
        fgq.fgq_quantize_act(xf, 8, q=qf, scale_out=sxf, ws=wsf)
        for G in (4, 64):
            codes, alpha, prep, prepd = layers[G]
            fgq.fgq_conv2d(q, 8, sx, (B, H, W, C), codes, alpha, O, R, S, 1, 1, G, prepared=prep, y=outs[f"y{G}"])
            fgq.fgq_conv2d_dfp(q, 8, sx, (B, H, W, C), codes, prepd, O, R, S, 1, 1, G, out=outs[f"yd{G}"])
        codes, alpha, prep, _ = layers[4]
        fgq.fgq_conv2d_q(q, 8, sx, (B, H, W, C), codes, alpha, O, R, S, 1, 1, 4, 8, osc, prepared=prep,
                         q_out=outs["q8"])
        fgq.fgq_gemm_ws(qf, 8, sxf, M, KF, cf, af, OF, GF, prepared=pf, out=outs["gf"], ws=wsg)
        fgq.fgq_gemm_dfp_ws(qf, 8, sxf, M, KF, cf, pfd, OF, GF, out=outs["gfd"], ws=wsgd)
        fgq.fgq_quantize_act(xr, 8, q=qr, scale_out=sxr, ws=wsr)
        fgq.fgq_conv2d(qr, 8, sxr, (BR, HR, HR, CR), cr, ar, OR, 1, 1, 1, 0, 4, prepared=pr, y=outs["yr"])
        fgq.fgq_conv2d_q(qr, 8, sxr, (BR, HR, HR, CR), cr, ar, OR, 1, 1, 1, 0, 4, 8, osc, prepared=pr,
                         q_out=outs["qr8"])

    step()
    torch.cuda.synchronize()
    eager = {k: v.clone() for k, v in outs.items()}
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step()
    for rep in range(3):
        for v in outs.values():
            v.zero_()
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for k, v in outs.items():
            assert torch.equal(v, eager[k]), f"replay {rep}: {k} differs from the eager result"
        step()  # eager work between replays
        torch.cuda.synchronize()
        for k, v in outs.items():
            assert torch.equal(v, eager[k]), f"eager after replay {rep}: {k} differs"


@pytest.mark.parametrize("G,bits", [(4, 8), (64, 4)])
def test_concurrent_chains_match_eager(G, bits):
    """Independent batches as concurrent chains of one graph (the
    benchmark's timed form): eight buffer sets dealt over four chains forked
    from the capturing stream and joined back; every replay, with eager work
    in between, reproduces each set's eager codes, scale and output."""
    B, H, W, C, O, R, S = 4, 14, 14, 128, 128, 3, 3
    K = R * S * C
    w = fi.he_weights(O, C, R, S, "chains", G)
    codes, alpha, _ = fgq.fgq_ternarize(torch.from_numpy(w).cuda(), G)
    prep = fgq.fgq_prepare_weights(codes, alpha, O, K, G)
    n = B * H * W * C
    sets = []
    for i in range(8):
        x = torch.from_numpy(fi.relu_gauss((n,), "chains-x", G, i)).cuda()
        sets.append(dict(x=x, q=torch.empty(n * bits // 8, dtype=torch.uint8, device="cuda"),
                         sx=torch.empty(1, device="cuda"),
                         ws=torch.empty(fgq.fgq_quantize_ws_bytes(n), dtype=torch.uint8, device="cuda"),
                         y=torch.empty((B, H, W, O), device="cuda")))

    def step(s):
        fgq.fgq_quantize_act(s["x"], bits, q=s["q"], scale_out=s["sx"], ws=s["ws"])
        fgq.fgq_conv2d(s["q"], bits, s["sx"], (B, H, W, C), codes, alpha, O, R, S, 1, 1, G, prepared=prep,
                       y=s["y"])

    for s in sets:
        step(s)
    torch.cuda.synchronize()
    eager = [{k: s[k].clone() for k in ("q", "sx", "y")} for s in sets]
    graph = torch.cuda.CUDAGraph()
    side = [torch.cuda.Stream() for _ in range(4)]
    with torch.cuda.graph(graph):
        cap = torch.cuda.current_stream()
        for st in side:
            st.wait_stream(cap)
        for r, st in enumerate(side):
            with torch.cuda.stream(st):
                for i in range(r, len(sets), len(side)):
                    step(sets[i])
        for st in side:
            cap.wait_stream(st)
    for rep in range(3):
        for s in sets:
            for k in ("q", "sx", "y"):
                s[k].zero_()
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for i, (s, e) in enumerate(zip(sets, eager)):
            for k in ("q", "sx", "y"):
                assert torch.equal(s[k], e[k]), f"replay {rep}: set {i} {k} differs from the eager result"
        step(sets[rep])  # eager work between replays
        torch.cuda.synchronize()
        assert torch.equal(sets[rep]["y"], eager[rep]["y"])
