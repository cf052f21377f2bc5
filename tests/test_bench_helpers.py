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


def test_summarize_trace_counts_blocks(tmp_path, capsys):
    """The trace summary cuts library kernels into blocks at idle gaps and
    counts each block's device-to-host copies (synthetic trace files in the
    column layout of rocprofv3's CSV output)."""
    import json
    import bench
    gap = bench.TRACE_GAP_S
    plan = {"gap_s": gap, "trace_blocks": [
        {"workload": "w", "mechanism": "resident", "invocations": 2, "T": 3,
         "library_counts_per_invocation": [1, 0]},
        {"workload": "w", "mechanism": "host_rt", "invocations": 2, "T": 3,
         "library_counts_per_invocation": [9, 3]}]}
    (tmp_path / "plan.out").write_text("noise\n" + json.dumps(plan) + "\n")
    rows = ["Kind,Kernel_Name,Start_Timestamp,End_Timestamp"]
    t = 10_000
    for _ in range(2):  # resident: one chain kernel per invocation
        rows.append("KERNEL_DISPATCH,rc_chain_kernel<32>,%d,%d" % (t, t + 5000))
        t += 6000
    rows.append("KERNEL_DISPATCH,rc_prep_kernel,%d,%d" % (t + 10, t + 20))  # not counted
    t += int(gap * 1e9)
    copies = ["Kind,Direction,Start_Timestamp,End_Timestamp"]
    for _ in range(2 * 3):  # host round trip: decide, copy, two bodies per step
        rows.append("KERNEL_DISPATCH,rc_decide_kernel<4>,%d,%d" % (t, t + 100))
        copies.append("MEMORY_COPY,MEMORY_COPY_DEVICE_TO_HOST,%d,%d" % (t + 150, t + 160))
        rows.append("KERNEL_DISPATCH,\"rc_body_kernel<32, true, true>\",%d,%d" % (t + 200, t + 300))
        rows.append("KERNEL_DISPATCH,\"rc_body_kernel<32, true, false>\",%d,%d" % (t + 300, t + 400))
        t += 10_000
    copies.append("MEMORY_COPY,MEMORY_COPY_HOST_TO_DEVICE,%d,%d" % (t - 5000, t - 4000))
    d = tmp_path / "trace"
    d.mkdir()
    (d / "x_kernel_trace.csv").write_text("\n".join(rows) + "\n")
    (d / "x_memory_copy_trace.csv").write_text("\n".join(copies) + "\n")
    blits = ["Kind,Kernel_Name,Start_Timestamp,End_Timestamp"]
    api = ["Domain,Function,Start_Timestamp,End_Timestamp"]
    for line in copies[1:]:
        t0 = int(line.split(",")[2])
        if "DEVICE_TO_HOST" in line:
            rows.append("KERNEL_DISPATCH,__amd_rocclr_copyBuffer,%d,%d" % (t0 + 1, t0 + 9))
            api.append("HIP_RUNTIME_API,hipMemcpyAsync,%d,%d" % (t0 - 50, t0 - 40))
    api.append("HIP_RUNTIME_API,hipLaunchKernel,%d,%d" % (t - 9000, t - 8990))
    (d / "x_kernel_trace.csv").write_text("\n".join(rows) + "\n")
    (d / "x_hip_api_trace.csv").write_text("\n".join(api) + "\n")
    bench.summarize_trace(str(d), str(tmp_path / "plan.out"))
    out = capsys.readouterr().out.strip().splitlines()
    assert out[2].startswith("| w | resident | 2 | 1.00 | 0.00 | 0.00 | 0.00 | (1, 0) |"), out[2]
    assert out[3].startswith("| w | host_rt | 2 | 9.00 | 3.00 | 3.00 | 3.00 | (9, 3) |"), out[3]


class _FakeSets:
    """Stand-in for bench.Sets: n buffer sets, no device memory."""

    def __init__(self, rc, n):
        self.sets = [(None, rc.RcBuffers(0x1000 * (i + 1), 0, 0, 0, 0, 0, 64)) for i in range(n)]

    def __getitem__(self, i):
        return self.sets[i % len(self.sets)][1]


def test_launch_table_and_step_clock():
    """The timing loops' pre-bound calls: invocation i uses buffer set
    i mod n_sets and cohort range i mod n_ranges (the table repeats after
    their least common multiple), and every call continues the step clock
    (step0 = invocations so far times T), across calls of the loop."""
    from paper_2608_12123_amd import rc_cohort as rc
    sets = _FakeSets(rc, 4)
    ranges = [(c, c + 1) for c in range(6)]
    calls = bench.Launches(rc, "handle", sets, 8, ranges, 0)
    assert len(calls.table) == 12
    for i, (b, cb, ce) in enumerate(calls.table):
        assert b._obj is sets[i % 4] and (cb, ce) == ranges[i % 6]
    seen = []
    calls.chain_fn = lambda h, b, step0, T, mode, cb, ce, st: seen.append((b._obj, step0, T, mode, cb, ce)) or 0
    base = bench._STEP_CLOCK[0]
    calls.chain(5, rc.RC_MODE_RESIDENT)
    calls.chain(3, rc.RC_MODE_HOST_ROUNDTRIP)
    assert [s[1] for s in seen] == [((base + i) * 8) & 0xFFFFFFFF for i in range(5)] + \
        [((base + 5 + i) * 8) & 0xFFFFFFFF for i in range(3)]
    assert [s[0] for s in seen[5:]] == [sets[0], sets[1], sets[2]]  # each loop starts at entry 0
    assert [s[3] for s in seen] == [rc.RC_MODE_RESIDENT] * 5 + [rc.RC_MODE_HOST_ROUNDTRIP] * 3
    calls.chain_fn = lambda *a: rc.RC_E_INVALID
    with pytest.raises(rc.RcError):
        calls.chain(1, rc.RC_MODE_RESIDENT)
