"""Pins for the oracle's activation quantization (Sec. 4: activations are
quantized to 8 or 4 bits before each convolution, one scale per tensor).

Checked through properties that any correct uniform unsigned quantizer with
scale max/qmax must satisfy, plus the packing order of 4-bit values.
"""
import numpy as np
import pytest

import fgq_inputs as fi
import oracle


@pytest.mark.parametrize("bits", [8, 4])
def test_quantizer_properties(bits):
    qmax = 255 if bits == 8 else 15
    x = fi.relu_gauss((3, 7, 5, 16), "qprop", bits).ravel()
    x[5] = -2.0  # a negative value (not produced by ReLU) clips to 0
    q, s = oracle.quantize_act(x, bits)
    vals = q if bits == 8 else np.stack([q & 15, q >> 4], 1).ravel()
    assert s == np.float32(x.max()) / np.float32(qmax)
    assert vals.max() == qmax and vals[np.argmax(x)] == qmax
    assert vals[5] == 0
    ok = x >= 0
    recon = vals.astype(np.float64) * np.float64(s)
    # round to nearest: within half a step (plus fp32 division rounding)
    assert np.all(np.abs(recon[ok] - x[ok].astype(np.float64)) <= 0.5 * s * (1 + 1e-5))
    # monotone
    order = np.argsort(x, kind="stable")
    assert np.all(np.diff(vals[order].astype(np.int64)) >= 0)
    # idempotent: quantizing the dequantized codes with the same scale
    q2, s2 = oracle.quantize_act((vals.astype(np.float32) * s), bits, scale=s)
    assert s2 == s
    np.testing.assert_array_equal(q2, q)


def test_u4_packing_order():
    x = np.array([1, 2, 3, 4, 15, 0, 7, 8], np.float32)
    q, s = oracle.quantize_act(x, 4, scale=1.0)
    assert list(q) == [0x21, 0x43, 0x0F, 0x87]  # even element in the low nibble


def test_scale_edge_cases():
    q, s = oracle.quantize_act(np.array([-1.0, -2.0, 0.0, -0.0], np.float32), 8)
    assert s == 1.0 and not q.any()
    q, s = oracle.quantize_act(np.array([0.0, 0.5, 1.0, 2.0], np.float32), 8, scale=0.5)
    assert s == 0.5 and list(q) == [0, 1, 2, 4]
    # ties round to even; values beyond qmax*s clip
    q, s = oracle.quantize_act(np.array([0.5, 1.5, 2.5, 300.0], np.float32), 8, scale=1.0)
    assert list(q) == [0, 2, 2, 255]
    q, s = oracle.quantize_act(np.array([np.nan, 1.0], np.float32), 8, scale=1.0)
    assert list(q) == [0, 1]
    with pytest.raises(oracle.OracleError) as e:
        oracle.quantize_act(np.ones(3, np.float32), 4)
    assert e.value.code == 4
    with pytest.raises(oracle.OracleError):
        oracle.quantize_act(np.ones(4, np.float32), 6)
