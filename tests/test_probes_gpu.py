"""The measurement aids run on the GPU and return PDEC_OK: the read-ceiling
probe (both modes) and the matrix/vector issue probe (every mode at 1, 2 and
4 waves per SIMD), small sizes."""
import pytest
import torch

from paper_2607_02963_amd import pdec

pytestmark = pytest.mark.gpu


def test_read_probe_runs():
    k = torch.ones(640, 4, 128, dtype=torch.bfloat16, device="cuda")
    v = torch.ones_like(k)
    for mode in (0, 1):
        sink = pdec.read_probe(k, v, mode, keys_per_item=128)
        torch.cuda.synchronize()
        assert int(sink.item()) == 0  # the sink is written only for a fixed hash value


@pytest.mark.parametrize("wps", [1, 2, 4])
def test_issue_probe_runs(wps):
    for mode in (0, 1, 2) + ((3,) if wps >= 2 else ()):
        sink = pdec.issue_probe(mode, wps, 16)
        torch.cuda.synchronize()
        assert float(sink.item()) == 0.0
