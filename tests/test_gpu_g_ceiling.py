"""The matrix-core ceiling measurement (nsp_mfma_ceiling) on the GPU: its
rate is the products it was asked for over its own time, within the nominal
peak, and zero operands (whose products toggle nothing) run at least as fast
as random ones."""
import pytest

from paper_2609_22755_amd import nsp

from gpu_util import require_gpu

pytestmark = pytest.mark.gpu

PEAK = 2516.6   # TFLOP/s: 256 CUs x 2.4 GHz x 4096 dense bf16 flop/clk


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


def test_ceiling_rates():
    import torch
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    products = 1 << 18
    rates = {}
    for zero in (False, True):
        for waves in (1, 2):
            sec, tf = nsp.nsp_mfma_ceiling(0, zero, waves, products)
            assert sec > 0
            assert tf == pytest.approx(products * cus * 4 * 32 * 32 * 16 * 2 / sec / 1e12, rel=1e-9)
            assert 0.2 * PEAK < tf < 1.02 * PEAK * cus / 256, (zero, waves, tf)
            rates[zero, waves] = tf
    for waves in (1, 2):
        assert rates[True, waves] >= 0.98 * rates[False, waves]
