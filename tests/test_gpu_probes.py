"""The calibration probes return plausible MI355X ceilings (the bench reports
the optimizer's rates against them)."""
import os
import sys

import pytest
import torch

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
import paper_2608_20818_amd as prm  # noqa: E402

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]


def test_peak_mfma_plausible():
    r = prm.peak_mfma(2000)
    print(r, flush=True)
    # dense bf16 spec is 2.5 PFLOP/s at 2.4 GHz; the power limit lowers the clock
    assert 300.0 < r["tflops"] < 2600.0
    assert 0.5 < r["clock_ghz"] < 2.6
    # executed FLOPs per cycle cannot exceed the 256 CUs x 4096 FLOP/cycle of the spec
    assert r["tflops"] * 1e12 / (r["clock_ghz"] * 1e9) <= 256 * 4096 * 1.02


def test_peak_hbm_plausible():
    r = prm.peak_hbm(256 << 20)
    print(r, flush=True)
    for k in ("read_gbs", "write_gbs", "copy_gbs", "rowwise_gbs"):
        assert 500.0 < r[k] < 8500.0, (k, r[k])
