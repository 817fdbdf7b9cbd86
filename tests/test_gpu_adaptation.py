"""GPU: per-level chunk sizes for the streaming adaptation come from the codec (C ABI), shrink as
the levels coarsen, and the study's rates are well formed."""
import dataclasses

import numpy as np
import pytest

from paper_2310_07240_amd import adaptation
from paper_2310_07240_amd import workloads as W
from gpu_helpers import say, torch_cuda

pytestmark = pytest.mark.gpu


def test_level_sizes_and_study_small():
    torch_cuda()
    w = dataclasses.replace(W.small(name="adapt_small", n_tokens=120, chunk_len=40, n_channels=64),
                            level_mult=adaptation.LEVELS, random_levels=False)
    sizes, errs = adaptation.level_sizes(w)
    say(f"sizes {sizes.tolist()} errs {errs}")
    assert sizes.shape == (3, len(adaptation.LEVELS))
    assert np.all(np.diff(sizes, axis=1) < 0)          # coarser bins, smaller payload
    # errors are reported as measured: a finer bin need not mean a smaller error, since deltas
    # beyond 127 bins are clamped (the finest level clamps more often)
    assert all(0.0 < e < 1.0 for e in errs)
    res = adaptation.study(sizes, errs, w.n_elem // 3, [1.0, 100.0], traces=20)
    for row in res:
        for k, v in row.items():
            if isinstance(v, dict):
                assert 0.0 <= v["slo_violation_rate"] <= 1.0
