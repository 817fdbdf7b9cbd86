"""The stream-layout study (paper_2310_07240_amd/layouts.py) on a small cache: both layouts
decode to the same fp16 cache, the stream counts follow their definitions, and the report's
figures are consistent."""
import pytest

from paper_2310_07240_amd import layouts
from paper_2310_07240_amd import workloads as W
from gpu_helpers import say

pytestmark = pytest.mark.gpu


def test_layout_study_small():
    w = W.small(name="layouts_small", n_ctx=2, n_layers=2, n_tokens=150, chunk_len=64,
                n_channels=96)
    r = layouts.run(w, reps=2)
    say(f"layouts: {r}")
    assert r["decodes_equal"]
    assert r["channel"]["streams"] == 2 * 3 * 2 * 2 * 96
    assert r["token"]["streams"] == 2 * 2 * 2 * 150
    for k in ("channel", "token"):
        assert r[k]["decode_ms"] > 0
        assert 0 < r[k]["payload_bits_per_element"] < 16
