"""The dense MFMA rate probe (a measurement aid beside the attention path):
it runs, reports the work of its launch, and leaves the sink untouched."""
import pytest
import torch

import paper_2609_32882_amd as vsa2

pytestmark = pytest.mark.gpu


def test_mfma_peak_probe_runs_and_counts():
    sink = torch.full((1,), 7.0, dtype=torch.float32, device="cuda")
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    st, flops = vsa2.vsa2_mfma_peak_probe(64, sink.data_ptr())
    torch.cuda.synchronize()
    assert vsa2.STATUS_NAMES[st] == "VSA2_OK"
    assert flops == cus * 16 * 4 * 64 * 2 * 32 * 32 * 16
    assert sink.item() == 7.0
    st, flops = vsa2.vsa2_mfma_peak_probe(0, None)
    assert vsa2.STATUS_NAMES[st] == "VSA2_OK" and flops == 0
