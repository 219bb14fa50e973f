"""The peak probes the benchmark reports (include/torpor_probe.h), at small sizes: each
returns a positive rate below what the hardware could possibly deliver."""
import pytest

import paper_2306_03622_amd as tp
from tests.common import torch_dev

pytestmark = pytest.mark.gpu


def test_peak_probes_small():
    torch_dev()
    tflops, clock = tp.probe_mfma_bf16(256, 64, 2)
    assert 1.0 < tflops < 2 * 2500.0
    assert 0.0 <= clock < 5.0
    hbm = tp.probe_hbm_read(64 << 20, 256, 2)
    assert 10.0 < hbm < 100000.0          # a 64 MiB buffer may partly come from the last-level cache
    gather = tp.probe_gather_h2d(16 << 20, 256, 2)
    assert 0.5 < gather < 200.0
