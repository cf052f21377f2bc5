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


def test_cohort_former_report_is_consistent():
    """The bench's cohort-share report (host code only): F <= P* <= U and
    A <= P* (every online batch is feasible), and the gap closure and the
    recovery are the ratios of those shares."""
    import bench
    from paper_2608_12123_amd import rc_cohort as rc
    from paper_2608_12123_amd import workload as wk
    d = bench.cohort_former(rc, wk, 25_000, ks=(32, 256), reps=1, seeds=(0,))
    for key, r in d["by_K"].items():
        assert r["F"] <= r["P_star"] <= r["U"] and r["A"] <= r["P_star"], (key, r)
        if r["U"] > r["F"]:
            assert abs(r["G"] - (r["P_star"] - r["F"]) / (r["U"] - r["F"])) < 1e-3
            assert 0.0 <= r["G"] <= 1.0
        if r["P_star"] > r["F"]:
            assert abs(r["R_A"] - (r["A"] - r["F"]) / (r["P_star"] - r["F"])) < 1e-3
            assert r["R_A"] <= 1.0
