"""GPU: the allocation-free quantization (fgq_quantize_act_noalloc, C ABI)
against fgq_quantize_act with a caller workspace: codes and scale bit for bit,
on two calls in a row, the second with a smaller input (the library's scratch
keeps the first call's partial maxima, which the second must not read), and
with a given scale."""
import ctypes

import numpy as np
import pytest
import torch

import fgq_inputs as fi

fgq = pytest.importorskip("paper_1705_01462_amd")

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr())


def with_ws(x, bits, scale_in=None):
    n = x.numel()
    q = torch.empty(n * bits // 8, dtype=torch.uint8, device="cuda")
    s = torch.empty(1, dtype=torch.float32, device="cuda")
    ws = torch.empty(max(fgq.fgq_quantize_ws_bytes(n), 4), dtype=torch.uint8, device="cuda")
    rc = fgq.lib().fgq_quantize_act(_ptr(x), n, bits, None if scale_in is None else _ptr(scale_in), _ptr(q),
                                    _ptr(s), _ptr(ws), ws.numel(),
                                    ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    assert rc == 0
    return q, s


def no_alloc(x, bits, scale_in=None):
    n = x.numel()
    q = torch.full((n * bits // 8,), 0xA5, dtype=torch.uint8, device="cuda")
    s = torch.full((1,), -1.0, dtype=torch.float32, device="cuda")
    rc = fgq.lib().fgq_quantize_act_noalloc(_ptr(x), n, bits, None if scale_in is None else _ptr(scale_in),
                                            _ptr(q), _ptr(s),
                                            ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    assert rc == 0, fgq.lib().fgq_status_string(rc)
    return q, s


@pytest.mark.parametrize("bits", [8, 4])
def test_no_alloc_matches_workspace_entry_point(bits):
    # the first input's maximum is far larger, so a stale partial maximum from
    # the first call would change every code of the second
    n1, n2 = 32 * 28 * 28 * 128, 3 * 17 * 17 * 64 + 2
    x1 = torch.from_numpy(fi.relu_gauss((n1,), "noalloc", 1) * np.float32(50.0)).cuda()
    x2 = torch.from_numpy(fi.relu_gauss((n2,), "noalloc", 2)).cuda()
    print(f"[noalloc] bits={bits} n1={n1} n2={n2}", flush=True)
    for x in (x1, x2):
        q_ref, s_ref = with_ws(x, bits)
        q, s = no_alloc(x, bits)
        torch.cuda.synchronize()
        assert s.item() == s_ref.item()
        assert torch.equal(q, q_ref)
    # a given scale (no scratch used)
    sc = torch.tensor([0.0123], dtype=torch.float32, device="cuda")
    q_ref, s_ref = with_ws(x2, bits, sc)
    q, s = no_alloc(x2, bits, sc)
    torch.cuda.synchronize()
    assert s.item() == s_ref.item() and torch.equal(q, q_ref)


def test_no_alloc_validation():
    L = fgq.lib()
    x = torch.zeros(64, dtype=torch.float32, device="cuda")
    q = torch.empty(64, dtype=torch.uint8, device="cuda")
    s = torch.empty(1, dtype=torch.float32, device="cuda")
    st = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    assert L.fgq_quantize_act_noalloc(None, 64, 8, None, _ptr(q), _ptr(s), st) == 1
    assert L.fgq_quantize_act_noalloc(_ptr(x), 64, 5, None, _ptr(q), _ptr(s), st) == 4
    assert L.fgq_quantize_act_noalloc(_ptr(x), 0, 8, None, _ptr(q), _ptr(s), st) == 2
    assert L.fgq_quantize_act_noalloc(_ptr(x), 63, 4, None, _ptr(q), _ptr(s), st) == 4
