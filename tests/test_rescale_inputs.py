"""The prefill rescale cases really exercise the rescale of live output.

For each case in :mod:`tests.softmax_rises`, the oracle's own scores (on
the CPU, after its own append and demotion) show query columns whose later
32-key unit rises more than 8 log2 units above every earlier unit's
maximum (plus a margin of 1 for the kernel's fp32 scores): a streaming
softmax with that threshold must rescale an accumulator that already
holds the first unit's output there.  The GPU parity of the same cases is
in test_gpu_prefill.py and test_gpu_fp8.py."""

import numpy as np
import pytest

from tests import softmax_rises as sr


@pytest.mark.parametrize("name", sorted(sr.CASES))
def test_case_forces_rescale_of_live_accumulators(name):
    case, hq, hkv, scale, dtype = sr.make(name)
    pool, bt, tags = sr.oracle_state(case, dtype)
    rises = sr.score_rises(case, pool, bt, tags, scale, dtype)
    firing = rises > 9.0
    print(f"{name}: {int(firing.sum())} of {rises.size} columns rise > 9 log2 units; max rise {rises.max():.1f}")
    assert firing.sum() >= 8
    assert rises.max() > 20.0
    if len(case["aligned"]):
        # every planted query column is among them
        for s, t, row, head in case["aligned"]:
            assert rises[row, head] > 9.0, (s, t, row, head)
