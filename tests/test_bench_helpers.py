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
