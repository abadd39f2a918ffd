"""GPU: a whole ResNet forward pass on the library, checked layer by layer.

ResNetChain (bench.py) runs every convolution and the fully-connected layer
as FGQ layers with their inputs quantized by fgq_quantize_act, each block's
shortcut addition and ReLU fused into its last convolution
(fgq_conv2d_residual; or, unfused, as torch ops after it), and the other
glue (max pooling, average pooling) in torch; the other ReLUs are the
quantizer's clamp at zero.  Chained layers cannot be compared with an
independently chained oracle (a one-ulp difference flips a rounding tie and
the chains diverge legitimately), so each layer is checked on the codes the
GPU fed it: its output against the oracle's layer on those codes (1e-5 of
the summand magnitude, bit-exact where the direct kernel ran; a block's
output against the oracle's last layer plus the shortcut and ReLU, within
that plus the addition's rounding), every quantization against the
oracle's quantization of the fp32 tensor it read, and the glue against
numpy on the GPU's own tensors.
"""
import numpy as np
import pytest
import torch

import bench
import fgq_inputs as fi
import oracle

fgq = pytest.importorskip("paper_1705_01462_amd")

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

TOL = 1e-5


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def maxpool3s2(a):
    """3x3 max pooling, stride 2, padding 1, of an NHWC array."""
    B, H, W, C = a.shape
    p = np.full((B, H + 2, W + 2, C), -np.inf, np.float32)
    p[:, 1:-1, 1:-1] = a
    Ho, Wo = (H - 1) // 2 + 1, (W - 1) // 2 + 1
    out = np.full((B, Ho, Wo, C), -np.inf, np.float32)
    for r in range(3):
        for s in range(3):
            out = np.maximum(out, p[:, r:r + 2 * Ho:2, s:s + 2 * Wo:2])
    return out


@pytest.mark.parametrize("depth,G,bits,hw,residual_fused", [(50, 4, 8, 64, True), (101, 64, 4, 32, True),
                                                             (50, 4, 8, 64, False)])
def test_chained_forward_layer_by_layer(depth, G, bits, hw, residual_fused):
    net = bench.ResNetChain(torch, fgq, fi, depth, G, bits, batch=2, hw=hw, tag="chain-test",
                            residual_fused=residual_fused)
    logits = host(net.forward())
    assert np.isfinite(logits).all()
    print(f"[chain] ResNet-{depth} G={G} u{bits} {hw}x{hw}: {len(net.layers)} layers", flush=True)

    def check_quant(src, e, name):
        q_ref, s_ref = oracle.quantize_act(host(src), bits)
        assert host(e["sx"])[0] == np.float32(s_ref), name
        np.testing.assert_array_equal(host(e["q"]), q_ref, err_msg=name)

    refs = {}
    for L in net.convs:
        name = L["name"]
        e = net.layers[name]
        B, H, W, C, O, R, S = (L[k] for k in ("B", "H", "W", "C", "O", "R", "S"))
        w = fi.he_weights(O, C, R, S, "chain-test", depth, name)
        if name == "conv1":
            w[:, 3:] = 0.0
        t, a, _ = oracle.ternarize(w, e["g"])
        q = host(e["q"])
        sx = host(e["sx"])[0]
        Ho, Wo = fgq.conv_out_hw(H, W, R, S, (L["stride"],) * 2, (L["pad"],) * 2)
        rows = np.arange(B * Ho * Wo, dtype=np.int64)
        y_ref, mag = oracle.conv2d_rows(q, bits, sx, (B, H, W, C), oracle.pack_codes(t), a, O, R, S,
                                        (L["stride"],) * 2, (L["pad"],) * 2, e["g"], rows)
        refs[name] = (y_ref, mag, e["prep"] is None)
        if residual_fused and name.endswith(".c3"):
            continue  # its output is the block's, checked below
        y = host(e["y"]).reshape(-1, O)
        err = np.abs(y.astype(np.float64) - y_ref)
        assert np.all(err <= TOL * mag), (name, float((err / np.maximum(mag, 1e-300)).max()))
        if e["prep"] is None:
            np.testing.assert_array_equal(y.view(np.uint32), y_ref.astype(np.float32).view(np.uint32))

    # the stem, the blocks and the head
    np.testing.assert_array_equal(host(net.stem), maxpool3s2(host(net.layers["conv1"]["y"])))
    h = net.stem
    for p, out in net.blocks.items():
        c1, c2, c3 = (net.layers[f"{p}.c{i}"] for i in (1, 2, 3))
        ds = net.layers.get(f"{p}.ds")
        check_quant(h, c1, p + ".c1")
        check_quant(c1["y"], c2, p + ".c2")
        check_quant(c2["y"], c3, p + ".c3")
        idn = host(ds["y"]) if ds is not None else host(h)
        if residual_fused:
            y_ref, mag, direct = refs[p + ".c3"]
            idn2 = idn.reshape(y_ref.shape)
            s = (y_ref + idn2).astype(np.float32)
            want = np.where(s < 0, np.float32(0), s)
            got = host(out).reshape(y_ref.shape)
            bound = TOL * mag + np.abs(y_ref.astype(np.float64) + idn2) * 2.0 ** -23
            if direct:
                np.testing.assert_array_equal(got, want, err_msg=p)
            assert np.all(np.abs(got.astype(np.float64) - want) <= bound), p
        else:
            np.testing.assert_array_equal(host(out), np.maximum(host(c3["y"]) + idn, np.float32(0)), err_msg=p)
        h = out
    np.testing.assert_allclose(host(net.pooled), host(h).mean(axis=(1, 2)), rtol=1e-6, atol=0)
    check_quant(net.pooled, net.layers["fc"], "fc")


def test_fused_forward_matches_two_step_layers():
    """The fused form (fgq_conv2d_q writing the next layer's codes at the
    calibrated static scale, fgq_conv2d_residual_q writing the next block's
    input codes) gives the codes of the layer followed by a separate
    quantization at that scale, for every fused layer."""
    net = bench.ResNetChain(torch, fgq, fi, 50, 4, 8, batch=2, hw=64, tag="chain-test")
    net.calibrate()
    assert np.isfinite(host(net.forward(fused=True))).all()
    names = list(net.blocks)
    for k, p in enumerate(names):
        if k > 0:
            # the block input's codes, written by the previous block's last
            # convolution at this block's static scale
            a = net.layers[f"{p}.c1"]
            q2, _ = fgq.fgq_quantize_act(net.blocks[names[k - 1]].reshape(-1), 8, scale_in=a["sx_static"])
            np.testing.assert_array_equal(host(a["q"]), host(q2), err_msg=f"{p}.c1")
    for k, p in enumerate(names):
        for i, j in ((1, 2), (2, 3)):
            e, nxt = net.layers[f"{p}.c{i}"], net.layers[f"{p}.c{j}"]
            sx = e["sx_static"] if (i == 2 or k > 0) else None
            net._conv(e, sx=sx)  # the same layer, fp32 output
            q2, _ = fgq.fgq_quantize_act(e["y"], 8, scale_in=nxt["sx_static"])
            np.testing.assert_array_equal(host(nxt["q"]), host(q2), err_msg=f"{p}.c{j}")


@pytest.mark.parametrize("depth,G,bits,hw", [(50, 4, 8, 64), (101, 64, 4, 32)])
def test_paper_pipeline_forward_layer_by_layer(depth, G, bits, hw):
    """The paper's pipeline (group scales as an 8-bit fixed point, the first
    layer at 8-bit weights): every layer bit-exact against the oracle's
    fixed-point layer on the codes the GPU fed it, each block output
    against the oracle's last layer plus the shortcut and ReLU, every
    quantization bit-exact; the fused form's codes equal the two-step ones."""
    net = bench.ResNetChain(torch, fgq, fi, depth, G, bits, batch=2, hw=hw, tag="chain-test", dfp=True)
    logits = host(net.forward())
    assert np.isfinite(logits).all()

    def check_quant(src, e, name):
        q_ref, s_ref = oracle.quantize_act(host(src), bits)
        assert host(e["sx"])[0] == np.float32(s_ref), name
        np.testing.assert_array_equal(host(e["q"]), q_ref, err_msg=name)

    refs = {}
    for L in net.convs:
        name = L["name"]
        e = net.layers[name]
        B, H, W, C, O, R, S = (L[k] for k in ("B", "H", "W", "C", "O", "R", "S"))
        w = fi.he_weights(O, C, R, S, "chain-test", depth, name)
        if name == "conv1":
            w[:, 3:] = 0.0
        q, sx = host(e["q"]), host(e["sx"])[0]
        st, pd = (L["stride"],) * 2, (L["pad"],) * 2
        if name == "conv1":
            W8, fl = oracle.w8_quantize(w)
            y_ref = oracle.conv2d_w8(q, bits, sx, (B, H, W, C), W8, fl, O, R, S, st, pd)
        else:
            t, a, _ = oracle.ternarize(w, e["g"])
            A, fl = oracle.dfp_alpha(a, 8)
            if name == "fc":
                y_ref = oracle.gemm_dfp(q, bits, sx, B, C, oracle.pack_codes(t), A, fl, O, e["g"])
            else:
                y_ref = oracle.conv2d_dfp(q, bits, sx, (B, H, W, C), oracle.pack_codes(t), A, fl, O, R, S, st, pd,
                                          e["g"])
        y_ref = y_ref.reshape(-1, O).astype(np.float32)
        refs[name] = y_ref
        if name.endswith(".c3"):
            continue  # its output is the block's, checked below
        np.testing.assert_array_equal(host(e["y"]).reshape(-1, O).view(np.uint32), y_ref.view(np.uint32),
                                      err_msg=name)

    np.testing.assert_array_equal(host(net.stem), maxpool3s2(host(net.layers["conv1"]["y"])))
    h = net.stem
    for p, out in net.blocks.items():
        c1, c2, c3 = (net.layers[f"{p}.c{i}"] for i in (1, 2, 3))
        ds = net.layers.get(f"{p}.ds")
        check_quant(h, c1, p + ".c1")
        check_quant(c1["y"], c2, p + ".c2")
        check_quant(c2["y"], c3, p + ".c3")
        idn = (host(ds["y"]) if ds is not None else host(h)).reshape(refs[p + ".c3"].shape)
        s = (refs[p + ".c3"] + idn).astype(np.float32)
        want = np.where(s < 0, np.float32(0), s)
        np.testing.assert_array_equal(host(out).reshape(want.shape).view(np.uint32), want.view(np.uint32),
                                      err_msg=p)
        h = out
    check_quant(net.pooled, net.layers["fc"], "fc")

    # the fused form: every fused layer's codes equal the layer then a separate quantization
    net.calibrate()
    assert np.isfinite(host(net.forward(fused=True))).all()
    names = list(net.blocks)
    for k, p in enumerate(names):
        if k > 0:
            a = net.layers[f"{p}.c1"]
            q2, _ = fgq.fgq_quantize_act(net.blocks[names[k - 1]].reshape(-1), bits, scale_in=a["sx_static"])
            np.testing.assert_array_equal(host(a["q"]), host(q2), err_msg=f"{p}.c1")
    for k, p in enumerate(names):
        for i, j in ((1, 2), (2, 3)):
            e, nxt = net.layers[f"{p}.c{i}"], net.layers[f"{p}.c{j}"]
            net._conv(e, sx=e["sx_static"] if (i == 2 or k > 0) else None)
            q2, _ = fgq.fgq_quantize_act(e["y"], bits, scale_in=nxt["sx_static"])
            np.testing.assert_array_equal(host(nxt["q"]), host(q2), err_msg=f"{p}.c{j}")


def maxpool3s2_valid(a):
    """3x3 max pooling, stride 2, no padding, of an NHWC array."""
    B, H, W, C = a.shape
    Ho, Wo = (H - 3) // 2 + 1, (W - 3) // 2 + 1
    out = np.full((B, Ho, Wo, C), -np.inf, np.float32)
    for r in range(3):
        for s in range(3):
            out = np.maximum(out, a[:, r:r + 2 * Ho:2, s:s + 2 * Wo:2])
    return out


@pytest.mark.parametrize("dfp", [False, True], ids=["fp32-scales", "paper-pipeline"])
def test_alexnet_forward_layer_by_layer(dfp):
    """AlexNet on the library, every layer checked on the codes the GPU fed
    it: against the oracle's layer (1e-5 of the summand magnitude with fp32
    group scales; bit-exact with fixed-point scales and the 8-bit-weight
    first layer), every quantization bit-exact, the pooling against numpy;
    the fused form's codes equal the layer then a separate quantization."""
    bits, G = 8, 4
    net = bench.AlexNetChain(torch, fgq, fi, G, bits, 2, tag="alexnet-test", dfp=dfp)
    assert np.isfinite(host(net.forward())).all()
    for L in net.convs:
        name = L["name"]
        e = net.layers[name]
        B, H, W, C, O, R, S = (L[k] for k in ("B", "H", "W", "C", "O", "R", "S"))
        w = fi.he_weights(O, C, R, S, "alexnet-test", name)
        if name == "conv1":
            w[:, 3:] = 0.0
        q, sx = host(e["q"]), host(e["sx"])[0]
        st, pd = (L["stride"],) * 2, (L["pad"],) * 2
        y = host(e["y"]).reshape(-1, O)
        t, a, _ = oracle.ternarize(w, e["g"])
        if dfp:
            if name == "conv1":
                W8, fl = oracle.w8_quantize(w)
                y_ref = oracle.conv2d_w8(q, bits, sx, (B, H, W, C), W8, fl, O, R, S, st, pd)
            else:
                A, fl = oracle.dfp_alpha(a, 8)
                y_ref = oracle.conv2d_dfp(q, bits, sx, (B, H, W, C), oracle.pack_codes(t), A, fl, O, R, S, st, pd,
                                          e["g"])
            np.testing.assert_array_equal(y.view(np.uint32), y_ref.reshape(-1, O).astype(np.float32).view(np.uint32),
                                          err_msg=name)
        else:
            rows = np.arange(y.shape[0], dtype=np.int64)
            y_ref, mag = oracle.conv2d_rows(q, bits, sx, (B, H, W, C), oracle.pack_codes(t), a, O, R, S, st, pd,
                                            e["g"], rows)
            assert np.all(np.abs(y.astype(np.float64) - y_ref) <= TOL * mag), name
    # pooling and the quantization of every layer input
    Ls = net.layers
    for a, b in (("conv1", "conv2"), ("conv2", "conv3"), ("conv5", "fc6")):
        np.testing.assert_array_equal(host(net.pooled[a]), maxpool3s2_valid(host(Ls[a]["y"])), err_msg=a)
        q_ref, s_ref = oracle.quantize_act(host(net.pooled[a]), bits)
        np.testing.assert_array_equal(host(Ls[b]["q"]), q_ref, err_msg=b)
    for a, b in (("conv3", "conv4"), ("conv4", "conv5"), ("fc6", "fc7"), ("fc7", "fc8")):
        q_ref, s_ref = oracle.quantize_act(host(Ls[a]["y"]), bits)
        assert host(Ls[b]["sx"])[0] == np.float32(s_ref), b
        np.testing.assert_array_equal(host(Ls[b]["q"]), q_ref, err_msg=b)
    # the fused form
    net.calibrate()
    assert np.isfinite(host(net.forward(fused=True))).all()
    for i, (a, b) in enumerate((("conv3", "conv4"), ("conv4", "conv5"), ("fc6", "fc7"), ("fc7", "fc8"))):
        e = Ls[a]
        net._layer(e, sx=e["sx_static"] if i in (1, 3) else None)  # the same layer, fp32 output
        q2, _ = fgq.fgq_quantize_act(e["y"], bits, scale_in=Ls[b]["sx_static"])
        np.testing.assert_array_equal(host(Ls[b]["q"]), host(q2), err_msg=b)
