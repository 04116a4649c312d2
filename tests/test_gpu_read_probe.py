"""The read-bandwidth calibration (cmoe_read_probe): a plausible rate for a
1 GiB buffer, between a tenth of the datasheet peak and the peak itself."""
import pytest

from gpu_util import say

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def test_read_probe_rate_is_plausible():
    from paper_2609_04895_amd import cmoe as B
    buf = torch.empty(1 << 30, dtype=torch.uint8, device="cuda:0")
    say("read probe: 1 GiB, 3 launches")
    gbs = B.cmoe_read_probe(buf, reps=3)
    say(f"read probe: {gbs:.0f} GB/s")
    assert 800.0 < gbs < 8000.0
    del buf
    torch.cuda.empty_cache()
