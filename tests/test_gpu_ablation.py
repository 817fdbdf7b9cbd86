"""GPU: the codec ablation (paper_2310_07240_amd.ablation) runs every configuration through the
C ABI on the tiny workload; the error of each decoded cache stays within its quantizer's bound."""
import pytest

from paper_2310_07240_amd import ablation
from paper_2310_07240_amd import workloads as W
from gpu_helpers import say, torch_cuda

pytestmark = pytest.mark.gpu


def test_ablation_tiny():
    torch_cuda()
    rows = ablation.run(W.TINY)
    for r in rows:
        say(r)
    assert [r["config"] for r in rows] == [c[0] for c in ablation.LADDER]
    for r in rows:
        assert 0.0 < r["payload_bits_per_element"] < 18.1
        # per element at most half a step of the coarsest bin (1.5 s) plus fp16 rounding;
        # relative to the cache's RMS that is well under 5 %
        assert r["rel_rms_error"] < 0.05
    # the same quantizer with one global table costs at least as many bits as with one table
    # per (layer, K/V, channel) here (the tables are fitted to the data they code)
    assert rows[1]["payload_bits_per_element"] <= rows[0]["payload_bits_per_element"]
    assert rows[3]["payload_bits_per_element"] <= rows[4]["payload_bits_per_element"]
    # tables fitted on another context still code this one (every frequency is at least 1)
    assert rows[5]["rel_rms_error"] == rows[3]["rel_rms_error"]
