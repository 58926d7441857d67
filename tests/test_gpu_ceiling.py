"""The sustained-MFMA-rate diagnostic on the GPU: both instruction patterns
on both operand kinds return a rate above zero and not above the nominal
bf16 peak (2516.6 TFLOP/s at 2.4 GHz, the highest clock of the part)."""
import pytest

from paper_2608_02474_amd import api

from gpu_util import say

pytestmark = pytest.mark.gpu

PEAK = 2516.6


@pytest.mark.parametrize("pattern", ["attention", "gemm"])
@pytest.mark.parametrize("data", ["constant", "gaussian"])
def test_mfma_ceiling_in_range(pattern, data):
    say(f"mfma ceiling {pattern} {data}")
    r = api.mfma_ceiling(pattern, data, seconds=0.2)
    say(f"  {r:.1f} TFLOP/s ({r / PEAK:.3f} of the nominal peak)")
    assert 0.0 < r <= PEAK * 1.001
