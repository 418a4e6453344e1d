"""Offline cost calibration on the device: both data paths measured, and
the fitted cost model explains the measurements."""
import pytest
import torch

from paper_2606_29982_amd import calibrate as cal

pytestmark = pytest.mark.gpu


def test_calibration_on_device():
    print("calibrating HBM (expert FFN) and the host link", flush=True)
    res = cal.calibrate(torch.device("cuda:0"))
    hbm, link = res["hbm"], res["link"]
    print(hbm.as_dict(), link.as_dict(), res["samples"], flush=True)
    # degradation factors of a real device: above 1 (slower than nominal), not absurdly so
    assert 1.0 <= hbm.alpha < 3.0 and hbm.r2 > 0.98
    assert 1.0 <= link.alpha < 3.0 and link.r2 > 0.98
    # a whole R1 expert (88 MB) costs far more over the host link than from HBM
    assert link.cost_us(88080384) > 20 * hbm.cost_us(88080384)
