"""The benchmark's work and roofline arithmetic against the figures derived
independently from the layer shapes for the benchmark configurations:
algorithmic bytes and operations of the single layers, the vector-ALU floor
of the per-group epilogue, and the roofline sums and bytes of the two
network stacks (every distinct layer counted with its multiplicity); and
that a request for more than one GPU ends with a message, not a result."""
import math

import bench
import fgq_inputs as fi


def test_single_layer_bytes_and_ops():
    M, K, _, _ = bench.layer_dims(bench.LAYER)
    assert (M, K) == (25088, 1152)
    assert 2 * M * 128 * K == 7_398_752_256
    assert bench.algorithmic_bytes(bench.LAYER, 4, 8) == 3_211_264 + 36_864 + 147_456 + 12_845_056
    assert bench.algorithmic_bytes(bench.LAYER, 64, 8) == 3_211_264 + 36_864 + 9_216 + 12_845_056
    M1, K1, _, _ = bench.layer_dims(bench.LAYER_1X1)
    assert (M1, K1) == (100352, 256)
    assert 2 * M1 * 64 * K1 == 3_288_334_336
    assert bench.algorithmic_bytes(bench.LAYER_1X1, 64, 8) == 25_690_112 + 4_096 + 1_024 + 25_690_112
    # one byte per group scale for fixed-point scales, 8-bit outputs when fused
    assert bench.algorithmic_bytes(bench.LAYER, 4, 8, alpha_bytes=1) == 3_211_264 + 36_864 + 36_864 + 12_845_056
    assert bench.algorithmic_bytes(bench.LAYER, 4, 8, out_bits=8) == 3_211_264 + 36_864 + 147_456 + 3_211_264


def test_valu_floor_of_the_per_group_epilogue():
    # 2 * M * O * (K / G) / (64 lanes * 256 CUs * 2.4 GHz)
    assert math.isclose(bench.valu_floor_us(bench.LAYER, 64), 2.94, abs_tol=0.005)


def test_stack_rooflines():
    for depth, G, bits, roof_us, gbytes, nlayers in ((50, 4, 8, 453.8, 3.56, 54), (101, 64, 4, 615.6, 4.68, 105)):
        tot_us = tot_bytes = 0.0
        n = 0
        for L, count in bench.stack_layers(fi, depth, 64):
            g = G if L["C"] % G == 0 else 4
            _, nbytes, r = bench.stack_layer_roofline(L, g, bits)
            tot_us += count * r
            tot_bytes += count * nbytes
            n += count
        assert n == nlayers
        assert math.isclose(tot_us, roof_us, abs_tol=0.05), (depth, tot_us)
        assert math.isclose(tot_bytes / 1e9, gbytes, abs_tol=0.005), (depth, tot_bytes)


def test_more_than_one_gpu_exits_with_a_message():
    import os
    import subprocess
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    r = subprocess.run([sys.executable, os.path.join(root, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=300)
    assert r.returncode != 0
    assert "one GPU" in r.stdout + r.stderr
    assert r.stdout.strip() == "" or not r.stdout.lstrip().startswith("{")  # no result line
