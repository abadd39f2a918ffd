"""GPU parity of the row-walking folded kernel: short reductions over many row
tiles (1x1 layers with fp32 group scales, K <= 128, more than 64 channels and
at least two row tiles per workgroup), through the C ABI.

Each case is chosen so that the full batch takes that kernel, and checks:
  * sampled row ranges (first, middle, last: a ragged tail where M is not a
    multiple of the tile) against the oracle, within 1e-5 of the summand
    magnitude;
  * the whole output against the same layer run image by image (the rows of
    one image do not depend on the others, and one image is too few tiles
    for the row-walking kernel, so each call takes the one-tile kernel):
    bit for bit, since both kernels share the arithmetic;
  * the fused next-layer codes (8-bit, and 4-bit for even O) against
    fgq_quantize_act of the fp32 output with the same scale, and against
    the image-by-image fused calls: bit for bit.
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
ROWS = 128


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def takes_row_kernel(M, K, O):
    """The eligibility rule of the row-walking kernel, as documented."""
    if K > 128 or O <= 64:
        return False
    tiles = -(-O // 128) * -(-M // 64)
    return tiles >= 4 * torch.cuda.get_device_properties(0).multi_processor_count


CASES = [
    # B, H, W, C, O, G, bits
    (16, 56, 56, 64, 256, 4, 8),     # K = 64 (half a step, zero-padded), two channel tiles
    (24, 56, 56, 128, 128, 4, 4),    # K = 128, uint4
    (17, 55, 55, 96, 160, 8, 8),     # ragged M, partial second channel tile, K = 96
    (8, 112, 112, 16, 96, 4, 4),     # K = 16, one partial channel tile, uint4
    (12, 57, 57, 32, 200, 32, 8),    # ragged M and O, G = 32 (8-bit codes stored directly: O % 16 != 0)
    (24, 56, 56, 64, 99, 4, 8),      # odd O: every output stored directly from registers
]


def layer(case):
    B, H, W, C, O, G, bits = case
    w = fi.he_weights(O, C, 1, 1, "rows", case)
    x = fi.relu_gauss((B, H, W, C), "rows", case)
    codes, alpha, _ = fgq.fgq_ternarize(torch.from_numpy(w).cuda(), G)
    q, sx = fgq.fgq_quantize_act(torch.from_numpy(x).cuda(), bits)
    t, a, _ = oracle.ternarize(w, G)
    ref = dict(codes=oracle.pack_codes(t), a=a)
    ref["q"], ref["s"] = oracle.quantize_act(x, bits)
    np.testing.assert_array_equal(host(codes), ref["codes"])
    np.testing.assert_array_equal(host(q), ref["q"])
    assert sx.item() == ref["s"]
    prep = fgq.fgq_prepare_weights(codes, alpha, O, C, G)
    return codes, alpha, q, sx, prep, ref, x.shape


def run(case, codes, alpha, q, sx, prep, shape, out_bits=0, out_scale=None):
    B, H, W, C, O, G, bits = case
    if out_bits:
        return fgq.fgq_conv2d_q(q, bits, sx, shape, codes, alpha, O, 1, 1, 1, 0, G, out_bits, out_scale,
                                prepared=prep)
    return fgq.fgq_conv2d(q, bits, sx, shape, codes, alpha, O, 1, 1, 1, 0, G, prepared=prep)


@pytest.mark.parametrize("case", CASES, ids=[f"B{c[0]}-{c[1]}x{c[2]}-{c[3]}to{c[4]}-G{c[5]}-u{c[6]}"
                                             for c in CASES])
def test_row_kernel(case):
    B, H, W, C, O, G, bits = case
    print(f"[rows] {case}", flush=True)
    M = B * H * W
    assert takes_row_kernel(M, C, O)
    assert not takes_row_kernel(H * W, C, O)  # one image: the one-tile kernel
    per_img = H * W * C * bits // 8
    assert per_img % 16 == 0  # image slices keep the matrix-core alignment
    codes, alpha, q, sx, prep, ref, shape = layer(case)
    y = host(run(case, codes, alpha, q, sx, prep, shape)).reshape(-1, O)

    # sampled rows against the oracle
    for row0 in sorted({0, M // 2 - ROWS // 2, M - ROWS}):
        y_ref = oracle.conv2d(ref["q"], bits, ref["s"], shape, ref["codes"], ref["a"], O, 1, 1, (1, 1),
                              (0, 0), G, rows=(row0, ROWS))[row0:row0 + ROWS]
        P = oracle.group_sums_conv(ref["q"], bits, shape, ref["codes"], O, 1, 1, (1, 1), (0, 0), G,
                                   row0, ROWS).astype(np.float64)
        mag = float(ref["s"]) * np.einsum("mog,og->mo", np.abs(P), ref["a"].astype(np.float64))
        err = np.abs(y[row0:row0 + ROWS].astype(np.float64) - y_ref.astype(np.float64))
        assert not (err > TOL * mag).any(), f"rows [{row0}, {row0 + ROWS}) beyond 1e-5 of the summand magnitude"
        assert np.linalg.norm(err) <= TOL * np.linalg.norm(y_ref.astype(np.float64)) + 1e-30

    # the whole output against image-by-image calls of the one-tile kernel
    qb = q.reshape(B, -1)
    one = (1, H, W, C)
    for b in range(B):
        yb = host(run(case, codes, alpha, qb[b], sx, prep, one)).reshape(-1, O)
        np.testing.assert_array_equal(yb.view(np.uint32), y[b * H * W:(b + 1) * H * W].view(np.uint32),
                                      err_msg=f"image {b}")

    # fused next-layer codes
    y_dev = torch.from_numpy(y).cuda().reshape(-1)
    for ob in ((8, 4) if O % 2 == 0 else (8,)):  # 4-bit codes pair channels
        s_out = torch.tensor([0.8 * float(y.max()) / (2 ** ob - 1)], dtype=torch.float32, device="cuda")
        qf = run(case, codes, alpha, q, sx, prep, shape, ob, s_out).reshape(-1)
        q_two, _ = fgq.fgq_quantize_act(y_dev, ob, scale_in=s_out)
        assert torch.equal(qf, q_two), f"fused {ob}-bit codes differ from conv + quantize"
        qfb = qf.reshape(B, -1)
        for b in (0, B // 2, B - 1):
            qb1 = run(case, codes, alpha, qb[b], sx, prep, one, ob, s_out).reshape(-1)
            assert torch.equal(qb1, qfb[b]), f"fused {ob}-bit codes of image {b} differ from the one-tile kernel"
