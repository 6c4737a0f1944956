"""The issue-rate probe behind the bench line's instruction-mix floor
(lamp_issue_rates): every rate is measured, positive and plausible, and one
emulated 8-bit step (decode, two broadcast FMAs, rounding) costs more than
its broadcast FMAs alone."""
import math

import pytest
import torch

pytestmark = pytest.mark.gpu


def test_issue_rates_measured():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_39361_amd import lamp
    r = lamp.issue_rates()
    print(r, flush=True)
    assert set(r) == set(lamp.ISSUE_RATE_KINDS)
    for k, v in r.items():
        assert math.isfinite(v) and 0.1 < v < 1000.0, (k, v)
    assert r["emulated_step"] > 2.0 * r["fmac_f32_dpp"]
