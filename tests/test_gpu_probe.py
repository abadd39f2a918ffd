"""The matrix-instruction rate probe (a measurement utility of the
benchmark): it runs, is deterministic, and rejects bad sizes before
launching anything."""
import pytest
import torch

fgq = pytest.importorskip("paper_1705_01462_amd")

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]


def test_probe_runs_and_is_deterministic():
    a = fgq.fgq_probe_mfma_i8(8, 16)
    b = fgq.fgq_probe_mfma_i8(8, 16)
    torch.cuda.synchronize()
    assert a.numel() == 8 * 256
    assert torch.equal(a, b)
    c = fgq.fgq_probe_mfma_i8(8, 17)
    torch.cuda.synchronize()
    assert not torch.equal(a, c)  # the rounds are not optimized away


def test_probe_rejects_bad_sizes():
    with pytest.raises(fgq.FgqError):
        fgq.fgq_probe_mfma_i8(0, 16)
    with pytest.raises(fgq.FgqError):
        fgq.fgq_probe_mfma_i8(4, 16, out=torch.empty(4 * 256 - 1, dtype=torch.int32, device="cuda"))
