"""The shader-clock probe that bench.py uses to state the peak at the clock a run actually had:
one workgroup per CU keeps the matrix cores busy; the clock it reads must lie between the
lowest DPM state and the published maximum, and the cycle count must match the MFMAs issued."""
import numpy as np
import pytest
import torch

from paper_2505_18654_amd import hstu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def test_clock_probe_reads_a_plausible_clock():
    blocks = torch.cuda.get_device_properties(0).multi_processor_count
    out = torch.zeros(3 * blocks, dtype=torch.int64, device="cuda")
    iters = 200_000
    khz = hstu.mtgr_debug_clock_probe(iters, blocks, out)
    torch.cuda.synchronize()
    o = out.view(blocks, 3).cpu().numpy().astype(np.float64)
    assert khz > 0 and (o[:, 1] > 0).all()
    mhz = o[:, 0] / o[:, 1] * khz / 1e3
    # 4 MFMAs of 32 cycles per iteration and wave, one wave per SIMD: at least that many cycles
    assert (o[:, 0] >= 0.95 * 4 * 32 * iters).all()
    assert 300 < float(np.median(mhz)) < 2600, mhz
