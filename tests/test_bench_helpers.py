"""Host helpers of bench.py, on the CPU."""
import numpy as np
import pytest

import bench
import oracle
from paper_2608_12123_amd import workload as wk


@pytest.mark.parametrize("key", ["tiny", "k256", "s100k"])
def test_decision_bitmap_read_back_from_effects(key):
    """The floor's bitmap, read back from an effect log, is the decision
    record the oracle keeps while it runs the chain."""
    wl = wk.WORKLOADS[key]
    inp = wk.make_inputs(wl, chunk=0) if wl.per_cohort_invocation else wk.make_inputs(wl)
    out = oracle.load().run_inputs(inp, n_steps=wl.n_steps, record=True)
    bits = bench.decisions_from_effects(out["eff_sid"], out["n_taken"], inp.cohort_offsets, inp.ld)
    assert np.array_equal(bits, out["decisions"])


def test_algorithmic_bytes_of_the_100k_workload():
    # state and outcome read and written once, 24 bytes per effect, counts
    assert bench.algorithmic_bytes(100000, 32, 16, 391) == 64825024
