"""Benchmark of the batched ready-cohort transition on one MI355X.

Default run (no flags): the 100,000-session workload (391 cohorts of K=256,
W=32, R=256, p=0.5, T=16 chained steps) -- the throughput / HBM-bandwidth
workload.  One bench step is one device-resident chain over all sessions
(every step of the hot path: route, decide, compact, update, emit, chain).
It prints ONE JSON line with the contract fields plus:

* ``roofline``: algorithmic bytes per launch of the resident chain kernel
  over its average duration, timed with HIP events on the launch stream,
  with the HBM traffic of the committed rocprofv3 counter summary;
  ``roofline_by_workload`` gives the same block (with its VALU busy
  fraction) for each single-launch workload: 100,000 and 1,000,000 sessions;
* ``valu``: VALU instructions per launch (committed SQ counter summary) and
  the fraction of the chip's VALU issue they occupy;
* ``host_roundtrip``: the same workload through the host-round-trip
  mechanism (4-byte readback + host branch + relaunch every chained step);
* ``floor``: the no-decision floor (decisions replayed from a bitmap);
* ``mechanisms``: resident, synchronized resident, floor and host round trip
  on all five workloads with the paper's row protocol (5 warmups, 3
  calibration samples, 30 rows of at least 100 ms each; median row in
  microseconds per invocation and per chained step, launches and
  device-to-host copies per invocation), beside the paper's own resident
  and host-round-trip medians (``mechanisms_paper_context``);
* ``cpu_baseline``: the single-threaded CPU oracle on the same workload, and
  the safe-suffix threshold K_r (batch sizes and chain lengths where the
  resident chain beats the oracle on one core and on all cores);
* ``cohort_former``: the cohort shares F, P*, U, the online share A and
  their ratios on seeded 1M-event arrival streams;
* ``hbm_measured`` and ``device``: measured copy and fill bandwidth and the
  device's properties, beside the spec peak.

Inputs are synthetic and seeded (see paper_2608_12123_amd/workload.py).  The
timed region rotates through enough buffer sets that the working set is
larger than the 256 MB Infinity Cache.  Before the W warmup steps, the
headline and roofline loops run 0.25 s of untimed resident chains so that
the timed launches run at steady clocks (``kernel_us.clock_warmup``).

Profiling modes: ``--profile-only`` (just the timed resident loop, for
counter runs), ``--copy-calibration`` (a plain copy of known size, the HBM
counter scale), ``--trace-mechanisms`` (resident and host-round-trip
invocation blocks on every workload, for a rocprofv3 kernel and memory-copy
trace) and ``--summarize-trace DIR PLAN`` (launches and device-to-host
copies per invocation from such a trace).
"""
from __future__ import annotations

import argparse
import json
import os
import platform
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = ("transitions/sec and µs per chained cohort step (resident vs host round trip); "
          "HBM GB/s")
HBM_PEAK_GBS = 8000.0
INFINITY_CACHE_BYTES = 256 << 20
PROFILE_TRAFFIC = os.path.join(ROOT, "profiles", "rc_chain_kernel_%s_traffic.txt")  # by workload
KERNEL_SRC = os.path.join(ROOT, "paper_2608_12123_amd", "csrc", "rc_cohort.hip")


def algorithmic_bytes(n_sessions, n_words, n_steps, n_cohorts):
    """Bytes the resident chain must move per launch: state and outcome read
    and written once per chain, one 24-byte effect per transition, and the
    per-cohort taken counts.  The route table (read from L2 into LDS) is not
    counted."""
    state = 2 * 4 * n_words * n_sessions
    outcome = 2 * 4 * n_sessions
    effects = 24 * n_sessions * n_steps
    counts = 4 * n_steps * n_cohorts
    return state + outcome + effects + counts


def kernel_src_hash():
    import hashlib
    with open(KERNEL_SRC, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def stored_traffic(workload_key):
    """HBM traffic per launch of the workload from the committed rocprofv3
    counter summary, valid only while the kernel source is unchanged."""
    path = PROFILE_TRAFFIC % workload_key
    if not os.path.exists(path):
        return None
    vals = {}
    with open(path) as f:
        for line in f:
            if "=" in line and not line.startswith("#"):
                k, v = line.split("=", 1)
                vals[k.strip()] = v.strip()
    if vals.get("kernel_src_sha256_16") != kernel_src_hash():
        return None
    try:
        return float(vals["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


PROFILE_VALU = os.path.join(ROOT, "profiles", "rc_chain_kernel_%s_valu.txt")  # by workload
ENGINE_CLOCK_HZ = 2.4e9  # MI355X peak engine clock


def stored_valu(workload_key):
    """VALU instructions per launch of the workload from the committed
    rocprofv3 counter summary, valid only while the kernel source is
    unchanged (None otherwise)."""
    path = PROFILE_VALU % workload_key
    if not os.path.exists(path):
        return None
    vals = {}
    with open(path) as f:
        for line in f:
            if "=" in line and not line.startswith("#"):
                k, v = line.split("=", 1)
                vals[k.strip()] = v.strip()
    if vals.get("kernel_src_sha256_16") != kernel_src_hash():
        return None
    try:
        return {"insts_per_launch": int(vals["SQ_INSTS_VALU"]), "waves": int(vals["SQ_WAVES"])}
    except (KeyError, ValueError):
        return None


class Sets:
    """Rotating device buffer sets for one handle."""

    def __init__(self, rc, inp, n_steps, n_sets):
        import torch
        self.inp = inp
        self.sets = []
        for _ in range(n_sets):
            t = {
                "state": torch.from_numpy(inp.state.view(np.int32)).cuda(),
                "outcome": torch.from_numpy(inp.outcome.view(np.int32)).cuda(),
                "eff_sid": torch.empty((n_steps, inp.ld), dtype=torch.int32, device="cuda"),
                "eff_tool": torch.empty((n_steps, inp.ld), dtype=torch.int32, device="cuda"),
                "eff_payload": torch.empty((n_steps, inp.ld, 4), dtype=torch.int32, device="cuda"),
                "n_taken": torch.empty((n_steps, inp.n_cohorts), dtype=torch.int32, device="cuda"),
            }
            self.sets.append((t, rc.buffers_of(t, inp.ld)))

    def bytes_per_set(self):
        return sum(v.numel() * 4 for v in self.sets[0][0].values())

    def __getitem__(self, i):
        return self.sets[i % len(self.sets)][1]

    def tensors(self, i):
        return self.sets[i % len(self.sets)][0]


def n_sets_for(bytes_per_set, min_total=2 * INFINITY_CACHE_BYTES, cap=16):
    return int(max(2, min(cap, -(-min_total // max(1, bytes_per_set)))))


# The step clock of the timing loops: every invocation continues the chain
# at the next T steps (step0 = invocations so far times T), as a serving loop
# that keeps stepping the same sessions would.  With step0 fixed at 0, a
# cohort stepped thousands of times falls into a cycle whose decisions repeat:
# the 32-session cohorts of the tiny workload end up all taken at every call,
# and the host round trip then never launches its not-taken body.
_STEP_CLOCK = [0]


def step_block(n):
    """Reserve n invocations on the step clock; returns the first one."""
    first = _STEP_CLOCK[0]
    _STEP_CLOCK[0] += n
    return first


def step0_next(T):
    return (step_block(1) * T) & 0xFFFFFFFF


class Launches:
    """Pre-bound calls of one handle for the timing loops.  Invocation i uses
    buffer set i mod n_sets and cohort range i mod n_ranges; those arguments
    are built once, and each call goes straight to the ctypes function the
    binding declares, so that a loop of small invocations spends no more host
    time per launch than the C ABI itself (a one-cohort tiny invocation is
    bound by that time)."""

    def __init__(self, rc, h, sets, T, ranges, stream, bits=None):
        import ctypes
        import math
        lib = rc.load_library()
        self.rc, self.h, self.T = rc, h, T
        self.chain_fn = lib.rc_cohort_run_chain
        self.floor_fn = lib.rc_cohort_run_floor
        self.stream = ctypes.c_void_p(stream)
        self.bits = ctypes.c_void_p(bits.data_ptr()) if bits is not None else None
        n_sets = len(sets.sets)
        n = n_sets * len(ranges) // math.gcd(n_sets, len(ranges))
        self.table = [(ctypes.byref(sets[i]),) + tuple(ranges[i % len(ranges)]) for i in range(n)]

    def chain(self, n, mode, sync_each=False):
        """n calls of rc_cohort_run_chain, table entries 0..n-1 (cyclic)."""
        import torch
        fn, h, T, st_h, tab = self.chain_fn, self.h, self.T, self.stream, self.table
        m, base = len(tab), step_block(n)
        sync = torch.cuda.current_stream().synchronize if sync_each else None
        for i in range(n):
            b, cb, ce = tab[i % m]
            st = fn(h, b, ((base + i) * T) & 0xFFFFFFFF, T, mode, cb, ce, st_h)
            if st:
                raise self.rc.RcError(st, "rc_cohort_run_chain")
            if sync:
                sync()

    def floor(self, n):
        """n calls of rc_cohort_run_floor with the bitmap given at build."""
        fn, h, T, st_h, tab, bits = self.floor_fn, self.h, self.T, self.stream, self.table, self.bits
        m = len(tab)
        for i in range(n):
            b, cb, ce = tab[i % m]
            st = fn(h, b, bits, T, cb, ce, st_h)
            if st:
                raise self.rc.RcError(st, "rc_cohort_run_floor")


def time_resident(rc, h, sets, inp, T, steps, warmup, stream, ranges=None, calls=None):
    """Pipelined resident chains.  Returns the wall seconds of the timed loop
    and its GPU time (ms) from one HIP event pair around it, recorded on the
    stream the kernels are launched on (the current torch stream, whose
    handle is passed to the library).  Nothing else is enqueued between the
    launches, so region time / steps is the average launch duration plus the
    small gap between back-to-back launches."""
    import torch
    calls = calls or Launches(rc, h, sets, T, ranges or [(0, inp.n_cohorts)], stream)
    cur = torch.cuda.current_stream()
    assert cur.cuda_stream == stream
    calls.chain(warmup, rc.RC_MODE_RESIDENT)
    r0, r1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    r0.record(cur)
    calls.chain(steps, rc.RC_MODE_RESIDENT)
    r1.record(cur)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    return wall, r0.elapsed_time(r1)


# After an idle spell the GPU takes a few tens of milliseconds of load to
# reach its steady clocks (a 2000-launch loop of the 100,000-session chain
# timed straight after set-up ran 9% slower than the same loop timed again).
# Before the W warmup steps, the headline and roofline loops therefore run
# untimed resident chains for CLOCK_WARMUP_S of wall time.
CLOCK_WARMUP_S = 0.25


def warm_calls(calls, mode, seconds=CLOCK_WARMUP_S):
    """Untimed calls (resident or host round trip by `mode`; the floor when
    mode is None), in blocks of about 5 ms, until `seconds` of wall time
    have passed.  Returns the calls made."""
    import torch
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    n, block = 0, 8
    while True:
        tb = time.perf_counter()
        if mode is None:
            calls.floor(block)
        else:
            calls.chain(block, mode)
        torch.cuda.synchronize()
        n += block
        now = time.perf_counter()
        if now - t0 >= seconds:
            return n
        block = int(max(1, min(4096, block * 0.005 / max(now - tb, 1e-6))))


def time_resident_synced(rc, h, sets, inp, T, steps, stream, ranges, calls=None):
    import torch
    calls = calls or Launches(rc, h, sets, T, ranges, stream)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    calls.chain(steps, rc.RC_MODE_RESIDENT, sync_each=True)
    return time.perf_counter() - t0


def decisions_from_effects(eff_sid, n_taken, offsets, ld):
    """The decision bitmap ([T][ceil(ld/32)] uint32) a chain made, read back
    from its effect log: within each cohort's slots the first n_taken[t][c]
    hold the taken sessions (the stable partition puts them first)."""
    T = eff_sid.shape[0]
    off = np.asarray(offsets, dtype=np.int64)
    sizes = np.diff(off)
    slot_rank = np.arange(off[-1]) - np.repeat(off[:-1], sizes)
    dec = np.zeros((T, ld), dtype=bool)
    for t in range(T):
        taken_slot = slot_rank < np.repeat(n_taken[t].astype(np.int64), sizes)
        dec[t, eff_sid[t, :off[-1]][taken_slot].astype(np.int64)] = True
    words = np.zeros((T, (ld + 31) // 32), dtype=np.uint64)
    for b in range(32):
        col = dec[:, b::32]
        words[:, :col.shape[1]] |= col.astype(np.uint64) << np.uint64(b)
    return words.astype(np.uint32)


def floor_bits(rc, h, inp, T, stream):
    """Device decision bitmap for the no-decision floor: the decisions one
    resident chain over every cohort makes on fresh inputs."""
    import torch
    one = Sets(rc, inp, T, 1)
    rc.rc_cohort_run_chain(h, one[0], 0, T, rc.RC_MODE_RESIDENT, 0, inp.n_cohorts, stream)
    torch.cuda.synchronize()
    t = one.tensors(0)
    bits = decisions_from_effects(t["eff_sid"].cpu().numpy().view(np.uint32),
                                  t["n_taken"].cpu().numpy().view(np.uint32),
                                  inp.cohort_offsets, inp.ld)
    return torch.from_numpy(bits.view(np.int32)).cuda()


def time_floor(rc, h, sets, bits, inp, T, steps, warmup, stream, ranges=None, calls=None):
    """Pipelined no-decision-floor launches (same protocol as the resident
    chain).  Returns the wall seconds of the timed loop."""
    import torch
    calls = calls or Launches(rc, h, sets, T, ranges or [(0, inp.n_cohorts)], stream, bits)
    calls.floor(warmup)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    calls.floor(steps)
    torch.cuda.synchronize()
    return time.perf_counter() - t0


def time_hrt(rc, h, sets, inp, T, steps, warmup, stream, ranges=None, calls=None):
    import torch
    calls = calls or Launches(rc, h, sets, T, ranges or [(0, inp.n_cohorts)], stream)
    calls.chain(warmup, rc.RC_MODE_HOST_ROUNDTRIP)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    calls.chain(steps, rc.RC_MODE_HOST_ROUNDTRIP)
    torch.cuda.synchronize()
    return time.perf_counter() - t0


# The paper's row protocol (Section 7 "Grid and independent unit"): per
# workload and mechanism, 5 warmup invocations, 3 calibration samples, then
# 30 timed rows of at least 100 ms of work each; the median row is reported.
MECH_WARMUPS = 5
MECH_CALIBRATION = 3
MECH_ROWS = 30
MECH_ROW_S = 0.100


def _calibrated_count(timed, row_s, first=10, min_sample_s=0.02):
    """Invocations per row so that a row takes at least row_s: the median
    per-invocation time of MECH_CALIBRATION samples, each grown until it
    takes at least min_sample_s, plus a 10% margin."""
    k = first
    while True:
        t = timed(k)
        if t >= min_sample_s or k >= 1 << 20:
            break
        k = int(k * max(2.0, 1.2 * min_sample_s / max(t, 1e-9)))
    per = float(np.median([t / k] + [timed(k) / k for _ in range(MECH_CALIBRATION - 1)]))
    return max(1, int(np.ceil(1.1 * row_s / max(per, 1e-9)))), per


def _rows(timed, n_per_row, rows, row_s=0.0):
    """Microseconds per invocation and milliseconds per row of `rows` timed
    rows of n_per_row invocations each: (median, 10th percentile, 90th
    percentile, median row ms, invocations per row).  Rows whose median
    falls short of row_s are timed again with a count scaled up to match."""
    for _ in range(3):
        secs = [timed(n_per_row) for _ in range(rows)]
        med = float(np.median(secs))
        if med >= row_s:
            break
        n_per_row = int(np.ceil(n_per_row * 1.05 * row_s / max(med, 1e-9)))
    us = [t / n_per_row * 1e6 for t in secs]
    return (float(np.median(us)), float(np.percentile(us, 10)), float(np.percentile(us, 90)),
            med * 1e3, n_per_row)


def mechanism_row(rc, wk, key, rows=MECH_ROWS, row_s=MECH_ROW_S, common_count=False):
    """Resident (pipelined and synchronized), no-decision floor and host
    round trip on one workload, invocations as the workload defines them, with
    the paper's row protocol.  Each mechanism's row count is calibrated on
    that mechanism so that every row holds at least row_s of its work; with
    common_count, every mechanism uses the count calibrated on the fastest
    one (the pipelined resident chain), as in the paper -- whose mechanisms
    differ by at most 2.4x, while here the host round trip is 4-42x slower,
    which makes its rows that much longer.  Single-launch workloads rotate
    enough buffer sets that a row streams from HBM, not from the 256 MB
    Infinity Cache."""
    import torch
    wl = wk.WORKLOADS[key]
    inp = wk.make_inputs(wl)
    T = wl.n_steps
    h = rc.rc_cohort_create(n_sessions=inp.n_sessions, n_words=inp.n_words, n_routes=inp.n_routes,
                            cohort_offsets=inp.cohort_offsets, table=inp.table,
                            route_mode=inp.route_mode, route_cdf=inp.route_cdf,
                            decide_thr=inp.decide_thr)
    try:
        if wl.per_cohort_invocation:
            ranges = [(c, c + 1) for c in range(inp.n_cohorts)]
            per_inv = wl.cohort_size * T
            n_sets = 1
        else:
            ranges = [(0, inp.n_cohorts)]
            per_inv = inp.n_sessions * T
            probe = Sets(rc, inp, T, 1)
            n_sets = n_sets_for(probe.bytes_per_set())
            del probe
        sets = Sets(rc, inp, T, n_sets)
        stream = torch.cuda.current_stream().cuda_stream
        bits = floor_bits(rc, h, inp, T, stream)
        calls = Launches(rc, h, sets, T, ranges, stream, bits)
        timers = {
            "resident": lambda k: time_resident(rc, h, sets, inp, T, k, 0, stream, ranges, calls)[0],
            "resident_synced": lambda k: time_resident_synced(rc, h, sets, inp, T, k, stream, ranges, calls),
            "floor": lambda k: time_floor(rc, h, sets, bits, inp, T, k, 0, stream, ranges, calls),
            "host_rt": lambda k: time_hrt(rc, h, sets, inp, T, k, 0, stream, ranges, calls),
        }
        res = {}
        counts = {}
        for name, timed in timers.items():
            timed(MECH_WARMUPS)
            n, _ = _calibrated_count(timed, row_s)
            counts[name] = n
        if common_count:
            counts = {name: counts["resident"] for name in counts}
        for name, timed in timers.items():
            res[name] = _rows(timed, counts[name], rows, 0.0 if common_count else row_s)
            counts[name] = res[name][4]
        rc.rc_cohort_run_chain(h, sets[0], step0_next(T), T, rc.RC_MODE_RESIDENT, *ranges[0], stream)
        res_counts = rc.rc_cohort_last_counts(h)
        rc.rc_cohort_run_chain(h, sets[0], step0_next(T), T, rc.RC_MODE_HOST_ROUNDTRIP, *ranges[0], stream)
        hrt_counts = rc.rc_cohort_last_counts(h)
        torch.cuda.synchronize()
        set_bytes = sets.bytes_per_set()
    finally:
        rc.rc_cohort_destroy(h)
    spread = lambda x: [round(x[1], 3), round(x[2], 3)]
    r_med, s_med, f_med, h_med = (res[k][0] for k in ("resident", "resident_synced", "floor", "host_rt"))
    return {
        "workload": wl.title, "T": T, "transitions_per_invocation": per_inv,
        "resident_us_per_invocation": round(r_med, 3),
        "resident_us_p10_p90": spread(res["resident"]),
        "resident_us_per_chained_step": round(r_med / T, 4),
        "resident_synced_us_per_invocation": round(s_med, 3),
        "resident_synced_us_p10_p90": spread(res["resident_synced"]),
        "host_rt_us_per_invocation": round(h_med, 3),
        "host_rt_us_p10_p90": spread(res["host_rt"]),
        "host_rt_us_per_chained_step": round(h_med / T, 4),
        "host_over_resident": round(h_med / r_med, 3),
        "host_over_resident_synced": round(h_med / s_med, 3),
        "floor_us_per_invocation": round(f_med, 3),
        "floor_us_p10_p90": spread(res["floor"]),
        "resident_over_floor": round(r_med / f_med, 3),
        "resident_transitions_per_s": round(per_inv / (r_med * 1e-6), 1),
        "host_rt_transitions_per_s": round(per_inv / (h_med * 1e-6), 1),
        "launches_per_invocation": {"resident": res_counts[0], "host_rt": hrt_counts[0]},
        "d2h_copies_per_invocation": {"resident": res_counts[1], "host_rt": hrt_counts[1]},
        "invocations_per_row": counts,
        "row_ms": {k: round(v[3], 2) for k, v in res.items()},
        "rows": rows, "warmups": MECH_WARMUPS, "calibration_samples": MECH_CALIBRATION,
        "common_count": common_count,
        "buffer_sets_rotated": n_sets, "bytes_per_buffer_set": set_bytes,
    }


def hbm_measured(n_bytes=512 << 20, reps=10):
    """Context for the roofline: what plain streaming kernels (torch's device
    copy and fill) reach on this GPU, timed with HIP events over `reps`
    dispatches of `n_bytes` each.  Copy counts bytes read plus bytes written."""
    import torch
    n = n_bytes // 4
    src = torch.ones(n, dtype=torch.int32, device="cuda")
    dst = torch.empty_like(src)
    out = {}
    for name, fn, moved in (("copy", lambda: dst.copy_(src), 2 * n_bytes),
                            ("fill", lambda: dst.fill_(7), n_bytes)):
        for _ in range(3):
            fn()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        out[name + "_GBps"] = round(moved * reps / (e0.elapsed_time(e1) * 1e-3) / 1e9, 1)
    out["bytes_per_dispatch"] = n_bytes
    out["note"] = ("torch device copy (read + write) and fill (write only) of 512 MiB; "
                   "context for the 8 TB/s spec peak, not the roofline peak")
    del src, dst
    return out


def cpu_model():
    """The host CPU's model name (Linux /proc/cpuinfo), else what platform
    reports."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or platform.machine()


# The paper's primary mechanism cell (Section 8 "Mechanism results", primary
# table): median over 30 rows of the batch-average wall time of one 32-epoch
# invocation (N = 256 agents, H = 32 chained epochs), one global decision
# per epoch over a 16-byte state, CUDA graphs, four NVIDIA placements.
PAPER_CONTEXT = {
    "what": "the paper's primary cell (N=256 agents, H=32 chained epochs, one global decision per "
            "epoch, 16-byte state, CUDA-graph mechanisms): median row us per 32-epoch invocation",
    "rows": [
        {"placement": "GTX 1660 Ti (local)", "resident_us": 273.0, "host_rt_us": 467.2,
         "host_over_resident": 1.71, "floor_us": 33.4},
        {"placement": "L4 (Modal)", "resident_us": 261.9, "host_rt_us": 625.3,
         "host_over_resident": 2.39, "floor_us": 39.7},
        {"placement": "L4 (RunPod)", "resident_us": 258.3, "host_rt_us": 533.3,
         "host_over_resident": 2.06, "floor_us": 37.3},
        {"placement": "H100 SXM5 (Lambda)", "resident_us": 309.0, "host_rt_us": 567.5,
         "host_over_resident": 1.84, "floor_us": 45.6},
    ],
    "ratio_range_all_cells": [1.19, 2.39],
    "note": "a different mechanism and hardware: context only, not a target",
}


def cpu_baseline(inp, T, min_seconds):
    """The oracle (plain single-threaded C) on the same workload, repeated
    until at least ``min_seconds`` of CPU work; also returns its outputs of
    the first repetition for the parity check of this run."""
    import oracle
    orc = oracle.load()
    reps, first = 0, None
    t0 = time.perf_counter()
    while True:
        out = orc.run_inputs(inp, n_steps=T)
        if first is None:
            first = out
        reps += 1
        el = time.perf_counter() - t0
        if el >= min_seconds:
            break
    trans = reps * inp.n_sessions * T
    return {"value": round(trans / el, 1), "unit": "transitions/s", "cores": 1, "kind": "oracle",
            "sample": "full workload (%d sessions x %d chained steps), %d repetition(s), %.1f s, "
                      "single thread, gcc -O2; host %s, %d logical CPUs"
                      % (inp.n_sessions, T, reps, el, cpu_model(), os.cpu_count() or 0),
            "cpu_model": cpu_model(), "host_logical_cpus": os.cpu_count() or 0}, first


def oracle_call_times(orc, inp, T, seconds, n_threads=1):
    """Seconds per call of the oracle's C entry point on preallocated buffers
    (one direct ctypes call per sample, no Python-side copies).  With
    n_threads > 1 the cohorts are split into that many contiguous ranges,
    each run by the unchanged oracle on its own host thread (ctypes releases
    the GIL; cohorts write disjoint outputs)."""
    import ctypes
    p32 = lambda a: a.ctypes.data_as(ctypes.POINTER(ctypes.c_uint32))
    state, outcome = inp.state.copy(), inp.outcome.copy()
    ld = state.shape[1]
    sid = np.zeros((T, ld), dtype=np.uint32)
    tool = np.zeros((T, ld), dtype=np.uint32)
    pay = np.zeros((T, ld, 4), dtype=np.uint32)
    cnt = np.zeros((T, inp.n_cohorts), dtype=np.uint32)
    off, tab = np.ascontiguousarray(inp.cohort_offsets), np.ascontiguousarray(inp.table).reshape(-1)
    cdf = None if inp.route_cdf is None else np.ascontiguousarray(inp.route_cdf)
    args = (inp.n_sessions, inp.n_words, inp.n_routes, inp.n_cohorts, p32(off), p32(tab),
            inp.route_mode, None if cdf is None else p32(cdf), inp.decide_thr, p32(state),
            p32(outcome), p32(sid), p32(tool), p32(pay), p32(cnt), ld, 0, T, 0, inp.n_cohorts, None)
    fn = orc.lib.rc_oracle_run_chain
    out = []
    t_end = time.perf_counter() + seconds
    if n_threads <= 1:
        while len(out) < 5 or time.perf_counter() < t_end:
            t0 = time.perf_counter()
            fn(*args)
            out.append(time.perf_counter() - t0)
        return out
    from concurrent.futures import ThreadPoolExecutor
    C = inp.n_cohorts
    cuts = [C * i // n_threads for i in range(n_threads + 1)]
    parts = [args[:18] + (cuts[i], cuts[i + 1], None) for i in range(n_threads) if cuts[i] < cuts[i + 1]]
    with ThreadPoolExecutor(len(parts)) as ex:
        while len(out) < 5 or time.perf_counter() < t_end:
            t0 = time.perf_counter()
            list(ex.map(lambda a: fn(*a), parts))
            out.append(time.perf_counter() - t0)
    return out


KR_SIZES = (32, 64, 128, 256, 512, 1024, 2048, 4096)
KR_STEPS = (1, 2, 4, 8, 16, 32)


def safe_suffix_threshold(rc, wk, sizes=KR_SIZES, steps=KR_STEPS, gpu_reps=200, cpu_seconds=0.05):
    """The hardware threshold K_r of the paper's model (Section 3, "Events and
    the hardware threshold"): the start of a measured safe suffix -- the
    smallest tested batch size from which every larger tested size is faster
    on the device-resident chain than on the named baseline, here the
    single-threaded oracle on the host cores, and an all-core bound.

    A batch of K sessions is one invocation over cohorts of min(K, 256)
    sessions (W = 32, R = 64 Zipf(1.1) routes, p = 0.3: the K = 256
    workload's shape), chained T steps.  GPU: median microseconds of one
    synchronized invocation (launch, run, stream sync: the latency an online
    caller sees).  CPU: median microseconds of the oracle on the same inputs;
    all cores: that time divided by min(cores, cohorts) -- perfect scaling
    over independent cohorts, an optimistic bound for the host, checked
    against a measured multi-threaded run at the largest K.  K_r is null
    when even the largest tested size is not faster."""
    import torch
    import oracle
    orc = oracle.load()
    stream = torch.cuda.current_stream().cuda_stream
    cores = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else (os.cpu_count() or 1)
    rows = []
    check = None
    for K in sizes:
        cs = min(K, 256)
        inp = wk.make_custom(n_words=32, n_routes=64, route_mode=wk.ROUTE_CDF, decide_thr=19661,
                             cohort_sizes=[cs] * (K // cs), n_steps=max(steps), seed_key=7000 + K)
        h = rc.rc_cohort_create(n_sessions=inp.n_sessions, n_words=32, n_routes=64,
                                cohort_offsets=inp.cohort_offsets, table=inp.table,
                                route_mode=inp.route_mode, route_cdf=inp.route_cdf,
                                decide_thr=inp.decide_thr)
        try:
            sets = Sets(rc, inp, max(steps), 1)
            for T in steps:
                for _ in range(10):
                    rc.rc_cohort_run_chain(h, sets[0], 0, T, rc.RC_MODE_RESIDENT, 0, inp.n_cohorts, stream)
                torch.cuda.synchronize()
                g = []
                for _ in range(gpu_reps):
                    t0 = time.perf_counter()
                    rc.rc_cohort_run_chain(h, sets[0], 0, T, rc.RC_MODE_RESIDENT, 0, inp.n_cohorts, stream)
                    torch.cuda.current_stream().synchronize()
                    g.append(time.perf_counter() - t0)
                c = float(np.median(oracle_call_times(orc, inp, T, cpu_seconds)))
                rows.append({"K": K, "T": T, "gpu_us": round(float(np.median(g)) * 1e6, 2),
                             "cpu_us": round(c * 1e6, 2),
                             "cpu_all_us": round(c / min(cores, inp.n_cohorts) * 1e6, 2)})
                if K == max(sizes) and T == 16:
                    n = min(cores, inp.n_cohorts)
                    m = float(np.median(oracle_call_times(orc, inp, T, 10 * cpu_seconds, n_threads=n)))
                    check = {"K": K, "T": T, "threads": n, "measured_us": round(m * 1e6, 2),
                             "bound_us": round(c / n * 1e6, 2)}
        finally:
            rc.rc_cohort_destroy(h)
    def threshold(key):
        k_r = {}
        for T in steps:
            r = sorted((x for x in rows if x["T"] == T), key=lambda x: x["K"])
            kr = None
            for x in reversed(r):
                if x["gpu_us"] < x[key]:
                    kr = x["K"]
                else:
                    break
            k_r[str(T)] = kr
        return k_r
    return {"k_r_by_T": threshold("cpu_us"), "k_r_by_T_all_cores": threshold("cpu_all_us"),
            "cores": cores, "all_core_check": check, "rows": rows,
            "note": "smallest tested K from which every larger tested K is faster on the resident "
                    "chain (synchronized invocation) than on the single-threaded oracle (k_r_by_T) "
                    "or on its all-core bound (k_r_by_T_all_cores); cohorts of min(K, 256) "
                    "sessions, W=32, R=64 Zipf(1.1), p=0.3"}


ONLINE_CAPACITY = 4096  # queue capacity per route of the online compactor


def cohort_former(rc, wk, latency_ns, ks=(32, 64, 128, 256), reps=3, seeds=(0, 1, 2)):
    """The library's cohort former and online compactor on the 1M-event
    Poisson arrival stream of the variable-cohort workload (Zipf routes,
    delta = the 50 ms launch deadline, one K for every route), for several
    independently seeded streams (chunks of the workload): the shares
    F <= P* <= U, the gap closure G = (P* - F) / (U - F), the online share A
    and its recovery R_A = (A - F) / (P* - F) -- G and R_A as the mean of the
    per-seed ratios -- and the host time of each call on the first stream
    (former: grouped sort, Algorithm 1 with witness, U; compactor: grouped
    sort and the policy sweep).  ``latency_ns`` is the launch-to-start
    latency the compactor budgets before each deadline."""
    wl = wk.WORKLOADS["s1m"]

    def best_of(fn):
        best, out = float("inf"), None
        for _ in range(reps):
            t0 = time.perf_counter()
            out = fn()
            best = min(best, time.perf_counter() - t0)
        return best, out

    per = {K: [] for K in ks}
    timing = {}
    for seed in seeds:
        times, routes, _ = wk.arrival_events(wl, chunk=seed)
        n = times.size
        for K in ks:
            k = np.full(wl.n_routes, K, dtype=np.uint32)
            pack = lambda: rc.rc_pack_shares(release_ns=times, route=routes, k_of_route=k,
                                             delta_ns=wk.DEADLINE_NS, witness=True)
            online = lambda: rc.rc_online_compact(release_ns=times, route=routes, k_of_route=k,
                                                  delta_ns=wk.DEADLINE_NS, latency_ns=latency_ns,
                                                  capacity=ONLINE_CAPACITY, witness=True)
            if seed == seeds[0]:
                t_pack, (res, _bat) = best_of(pack)
                t_on, (on, _b, _l) = best_of(online)
                timing[K] = (t_pack, t_on, n)
            else:
                res, _bat = pack()
                on, _b, _l = online()
            f, p, u = (res[x] / n for x in ("fixed_eligible", "packed", "overlap_eligible"))
            a = on["accelerated"] / n
            per[K].append({"F": f, "P_star": p, "U": u, "A": a,
                           "G": (p - f) / (u - f) if u > f else None,
                           "R_A": (a - f) / (p - f) if p > f else None,
                           "batches": res["n_batches"], "online_batches": on["n_batches"]})
    rows = {}
    for K in ks:
        v = per[K]
        mean = lambda key: (round(float(np.mean([x[key] for x in v if x[key] is not None])), 5)
                            if any(x[key] is not None for x in v) else None)
        t_pack, t_on, n = timing[K]
        rows["K%d" % K] = {
            "F": mean("F"), "P_star": mean("P_star"), "U": mean("U"), "A": mean("A"),
            "G": mean("G"), "R_A": mean("R_A"),
            "G_per_seed": [None if x["G"] is None else round(x["G"], 4) for x in v],
            "R_A_per_seed": [None if x["R_A"] is None else round(x["R_A"], 4) for x in v],
            "batches": v[0]["batches"], "online_batches": v[0]["online_batches"],
            "former_ms": round(t_pack * 1e3, 2), "compactor_ms": round(t_on * 1e3, 2),
            "former_events_per_s": round(n / t_pack, 1),
        }
    return {"events": wl.n_sessions, "routes": wl.n_routes, "delta_ms": wk.DEADLINE_NS / 1e6,
            "seeds": list(seeds), "online_latency_us": latency_ns / 1e3,
            "online_capacity": ONLINE_CAPACITY, "where": "host (library C++ code, one thread)",
            "by_K": rows}


def valu_of(key, k_avg_ms):
    """VALU instructions per launch of the workload's chain kernel (committed
    SQ counter summary) and the fraction of the chip's VALU issue they
    occupy over the measured kernel time; None when the summary is stale."""
    valu = stored_valu(key)
    if valu is None:
        return None
    import torch
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    busy = valu["insts_per_launch"] * 4.0 / (4 * cus * ENGINE_CLOCK_HZ * k_avg_ms * 1e-3)
    return {"insts_per_launch": valu["insts_per_launch"],
            "insts_per_wave": round(valu["insts_per_launch"] / valu["waves"], 1),
            "busy_frac": round(busy, 4),
            "basis": "SQ_INSTS_VALU (committed rocprofv3 summary) x 4 cycles / "
                     "(4 SIMDs x CUs x 2.4 GHz x measured kernel time)"}


def roofline_of(key, inp, T, k_avg_ms):
    """The HBM roofline block of one workload's resident chain kernel:
    algorithmic bytes per launch over the event-timed average launch."""
    abytes = algorithmic_bytes(inp.n_sessions, inp.n_words, T, inp.n_cohorts)
    achieved = abytes / (k_avg_ms * 1e-3) / 1e9
    traffic = stored_traffic(key)
    blk = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
           "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": traffic,
           "kernel": "rc_chain_kernel", "algorithmic_bytes_per_launch": abytes,
           "kernel_us": round(k_avg_ms * 1e3, 3)}
    if traffic is not None:
        blk["traffic_over_algorithmic"] = round(traffic / abytes, 4)
    valu = valu_of(key, k_avg_ms)
    if valu is not None:
        blk["valu"] = valu
    return blk


def measure_roofline(rc, wk, key, steps, warmup, warm=True):
    """Time `steps` resident launches of a single-launch workload (rotating
    buffer sets larger than the Infinity Cache) and return its roofline block."""
    import torch
    wl = wk.WORKLOADS[key]
    inp = wk.make_inputs(wl)
    T = wl.n_steps
    h = rc.rc_cohort_create(n_sessions=inp.n_sessions, n_words=inp.n_words, n_routes=inp.n_routes,
                            cohort_offsets=inp.cohort_offsets, table=inp.table,
                            route_mode=inp.route_mode, route_cdf=inp.route_cdf,
                            decide_thr=inp.decide_thr)
    try:
        probe = Sets(rc, inp, T, 1)
        n_sets = n_sets_for(probe.bytes_per_set())
        del probe
        sets = Sets(rc, inp, T, n_sets)
        stream = torch.cuda.current_stream().cuda_stream
        calls = Launches(rc, h, sets, T, [(0, inp.n_cohorts)], stream)
        n_warm = warm_calls(calls, rc.RC_MODE_RESIDENT) if warm else 0
        _, region_ms = time_resident(rc, h, sets, inp, T, steps, warmup, stream, calls=calls)
        blk = roofline_of(key, inp, T, region_ms / steps)
        blk.update({"workload": wl.title, "launches_timed": steps, "buffer_sets_rotated": n_sets,
                    "clock_warmup_launches": n_warm})
        return blk
    finally:
        torch.cuda.synchronize()
        rc.rc_cohort_destroy(h)


TRACE_GAP_S = 0.2  # idle time between the blocks of --trace-mechanisms


def trace_mechanisms(rc, wk, n=20):
    """For a kernel and memory-copy trace (rocprofv3): on every workload, n
    resident invocations, then n host-round-trip invocations, each block
    followed by TRACE_GAP_S of idle time so that --summarize-trace can cut
    the trace into blocks.  Prints the block plan as one JSON line."""
    import torch
    blocks = []
    stream = torch.cuda.current_stream().cuda_stream
    for key in wk.WORKLOAD_ORDER:
        wl = wk.WORKLOADS[key]
        inp = wk.make_inputs(wl)
        T = wl.n_steps
        h = rc.rc_cohort_create(n_sessions=inp.n_sessions, n_words=inp.n_words, n_routes=inp.n_routes,
                                cohort_offsets=inp.cohort_offsets, table=inp.table,
                                route_mode=inp.route_mode, route_cdf=inp.route_cdf,
                                decide_thr=inp.decide_thr)
        try:
            sets = Sets(rc, inp, T, 1)
            ranges = ([(c, c + 1) for c in range(inp.n_cohorts)] if wl.per_cohort_invocation
                      else [(0, inp.n_cohorts)])
            torch.cuda.synchronize()
            time.sleep(TRACE_GAP_S)
            for mech, mode in (("resident", rc.RC_MODE_RESIDENT), ("host_rt", rc.RC_MODE_HOST_ROUNDTRIP)):
                for i in range(n):
                    cb, ce = ranges[i % len(ranges)]
                    rc.rc_cohort_run_chain(h, sets[0], step0_next(T), T, mode, cb, ce, stream)
                counts = rc.rc_cohort_last_counts(h)
                torch.cuda.synchronize()
                time.sleep(TRACE_GAP_S)
                blocks.append({"workload": key, "mechanism": mech, "invocations": n, "T": T,
                               "library_counts_per_invocation": list(counts)})
        finally:
            rc.rc_cohort_destroy(h)
    print(json.dumps({"trace_blocks": blocks, "gap_s": TRACE_GAP_S}), flush=True)


def summarize_trace(trace_dir, plan_path):
    """Launches and device-to-host copies per invocation from a rocprofv3
    trace (--kernel-trace --hip-trace --memory-copy-trace) of
    --trace-mechanisms.  The library's chain-step kernels (chain, decide,
    body, counter clear) are cut into blocks at idle gaps longer than half of
    TRACE_GAP_S; in each block's time window (from half a gap before its first
    kernel to a quarter gap after its last) it counts the runtime's copy
    kernels (small device-to-host copies into pinned memory run as
    __amd_rocclr_copyBuffer), the hipMemcpy* calls of the HIP API trace and
    the SDMA device-to-host copies of the memory-copy trace.  Prints a
    markdown table."""
    import csv
    import glob

    def rows(pattern):
        out = []
        for path in sorted(glob.glob(os.path.join(trace_dir, "**", pattern), recursive=True)):
            out.extend(csv.DictReader(open(path)))
        return out

    plan = None
    with open(plan_path) as f:
        for line in f:
            if line.startswith("{") and "trace_blocks" in line:
                plan = json.loads(line)
    lib_kernels = ("rc_chain_kernel", "rc_decide_kernel", "rc_body_kernel", "rc_clear_kernel")
    ev, blit = [], []
    for r in rows("*kernel_trace.csv"):
        name = r.get("Kernel_Name", "")
        t0, t1 = int(r["Start_Timestamp"]), int(r["End_Timestamp"])
        if any(k in name for k in lib_kernels):
            ev.append((t0, t1, name))
        elif "copyBuffer" in name:
            blit.append(t0)
    ev.sort()
    api = [int(r["Start_Timestamp"]) for r in rows("*hip_api_trace.csv")
           if r.get("Function", "").startswith("hipMemcpy")]
    sdma = [int(r["Start_Timestamp"]) for r in rows("*memory_copy_trace.csv")
            if "DEVICE_TO_HOST" in r.get("Direction", "")]
    gap_ns = plan["gap_s"] * 1e9
    segs = []
    for e in ev:
        if segs and e[0] - segs[-1]["end"] < gap_ns / 2:
            segs[-1]["ev"].append(e)
            segs[-1]["end"] = max(segs[-1]["end"], e[1])
        else:
            segs.append({"start": e[0], "end": e[1], "ev": [e]})
    blocks = plan["trace_blocks"]
    if len(segs) != len(blocks):
        raise SystemExit("trace has %d kernel blocks, the plan %d" % (len(segs), len(blocks)))
    lines = ["| Workload | Mechanism | Invocations | Library kernel dispatches | Copy-kernel dispatches "
             "| hipMemcpy calls | SDMA D2H copies | Library's own counts (launches, D2H) "
             "| Mean chain-kernel us |", "|---|---|---|---|---|---|---|---|---|"]
    for seg, b in zip(segs, blocks):
        n = b["invocations"]
        lo, hi = seg["start"] - gap_ns / 2, seg["end"] + gap_ns / 4
        inside = lambda ts: sum(1 for t in ts if lo <= t <= hi) / n
        chain = [e[1] - e[0] for e in seg["ev"] if "rc_chain_kernel" in e[2]]
        lines.append("| %s | %s | %d | %.2f | %.2f | %.2f | %.2f | %s | %s |" % (
            b["workload"], b["mechanism"], n, len(seg["ev"]) / n, inside(blit), inside(api),
            inside(sdma), tuple(b["library_counts_per_invocation"]),
            "%.2f" % (sum(chain) / len(chain) / 1e3) if chain else "-"))
    lines.append("")
    lines.append("Per invocation (counts divided by the block's invocations).")
    print("\n".join(lines))


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=2000)
    ap.add_argument("--warmup", type=int, default=50)
    ap.add_argument("--workload", default="s100k",
                    help="workload of the headline line (tiny, k64, k256, s100k, s1m)")
    ap.add_argument("--hrt-steps", type=int, default=200)
    ap.add_argument("--no-mechanisms", action="store_true", help="skip the five-workload table")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-kr", action="store_true", help="skip the safe-suffix K_r sweep")
    ap.add_argument("--no-former", action="store_true", help="skip the cohort-former shares")
    ap.add_argument("--profile-only", action="store_true",
                    help="only the resident timed loop (for rocprofv3 counter runs)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only a plain device-to-device copy of known size (HBM counter scale)")
    ap.add_argument("--roofline-workloads", default="s100k,s1m",
                    help="single-launch workloads given a roofline block beside the headline")
    ap.add_argument("--mech-rows", type=int, default=MECH_ROWS)
    ap.add_argument("--mech-row-ms", type=float, default=MECH_ROW_S * 1e3)
    ap.add_argument("--mech-common-count", action="store_true",
                    help="one invocation count per workload for every mechanism, calibrated on the "
                         "fastest (the paper's protocol; the host-round-trip rows get long)")
    ap.add_argument("--trace-mechanisms", action="store_true",
                    help="only the block sequence for a kernel + memory-copy trace (rocprofv3)")
    ap.add_argument("--summarize-trace", nargs=2, metavar=("TRACE_DIR", "PLAN_OUTPUT"),
                    help="summarize a rocprofv3 trace of --trace-mechanisms and exit")
    args = ap.parse_args()

    if args.summarize_trace:
        summarize_trace(*args.summarize_trace)
        return

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(cohorts are independent, so sharding them over GPUs needs no "
              "collective). Run with --gpus 1.",
              file=sys.stderr)
        sys.exit(2)

    import torch

    if args.copy_calibration:
        n = 128 << 20  # 512 MiB of int32
        src = torch.ones(n, dtype=torch.int32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes_read_per_dispatch": n * 4,
                          "bytes_written_per_dispatch": n * 4, "dispatches": 5}), flush=True)
        return

    from paper_2608_12123_amd import rc_cohort as rc
    from paper_2608_12123_amd import workload as wk

    if not torch.cuda.is_available():
        sys.exit("bench.py needs an MI355X: no GPU is visible")
    rc.load_library()
    if args.trace_mechanisms:
        trace_mechanisms(rc, wk)
        return
    wl = wk.WORKLOADS[args.workload]
    inp = wk.make_inputs(wl)
    T = wl.n_steps
    N, C, W = inp.n_sessions, inp.n_cohorts, inp.n_words
    h = rc.rc_cohort_create(n_sessions=N, n_words=W, n_routes=inp.n_routes,
                            cohort_offsets=inp.cohort_offsets, table=inp.table,
                            route_mode=inp.route_mode, route_cdf=inp.route_cdf,
                            decide_thr=inp.decide_thr)
    stream = torch.cuda.current_stream().cuda_stream
    probe = Sets(rc, inp, T, 1)
    n_sets = n_sets_for(probe.bytes_per_set())
    del probe
    sets = Sets(rc, inp, T, n_sets)
    plan = rc.rc_cohort_plan_info(h)

    # parity of this run's kernel on fresh inputs against the oracle
    verified = None
    cpu = None
    if not args.profile_only and not args.no_cpu_baseline:
        cpu, want = cpu_baseline(inp, T, args.cpu_seconds)
        rc.rc_cohort_run_chain(h, sets[0], 0, T, rc.RC_MODE_RESIDENT, 0, C, stream)
        torch.cuda.synchronize()
        t = sets.tensors(0)
        verified = all(np.array_equal(t[k].cpu().numpy().view(np.uint32), want[k]) for k in want)
        sets = Sets(rc, inp, T, n_sets)  # fresh inputs again

    calls = Launches(rc, h, sets, T, [(0, C)], stream)
    n_warm = 0 if args.profile_only else warm_calls(calls, rc.RC_MODE_RESIDENT)
    wall, region_ms = time_resident(rc, h, sets, inp, T, args.steps, args.warmup, stream, calls=calls)
    trans_per_step = N * T
    value = trans_per_step * args.steps / wall
    ms_per_step = wall / args.steps * 1e3
    k_avg_ms = region_ms / args.steps
    roof = roofline_of(wl.key, inp, T, k_avg_ms)
    out = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "transitions/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 6),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u32",
        "data": "synthetic (seeded SplitMix64 inputs; no trace data)",
        "config": {
            "workload": wl.title, "sessions": N, "cohorts": C, "W": W, "R": inp.n_routes,
            "route_map": "mod" if inp.route_mode == wk.ROUTE_MOD else "zipf-cdf",
            "decide_thr": inp.decide_thr, "T": T, "mode": "device-resident chain",
            "parallelism": "single GPU", "buffer_sets_rotated": n_sets,
            "plan": {"workgroups": plan[0], "lanes_per_workgroup": plan[1], "idle_lanes": plan[2]},
        },
        "us_per_chained_step": round(ms_per_step * 1e3 / T, 4),
        "kernel_us": {"avg": round(k_avg_ms * 1e3, 3),
                      "timing": "one HIP event pair on the launch stream around the timed "
                                "loop, divided by the launches",
                      "clock_warmup": {"seconds": CLOCK_WARMUP_S if n_warm else 0,
                                       "launches": n_warm,
                                       "note": "untimed resident chains before the warmup steps, "
                                               "so that the timed loop runs at steady clocks"}},
        "roofline": {k: v for k, v in roof.items() if k != "valu"},
        "verified_vs_oracle": verified,
    }
    if "valu" in roof:
        out["valu"] = roof["valu"]
    by_wl = {}
    for key in [k for k in args.roofline_workloads.split(",") if k]:
        if key == wl.key:
            by_wl[key] = dict(roof, workload=wl.title, launches_timed=args.steps,
                              buffer_sets_rotated=n_sets, clock_warmup_launches=n_warm)
        else:
            by_wl[key] = measure_roofline(rc, wk, key, max(10, min(args.steps, 500)), min(args.warmup, 10),
                                          warm=not args.profile_only)
    if by_wl:
        out["roofline_by_workload"] = by_wl
    if not args.profile_only:
        hs = max(5, min(args.hrt_steps, args.steps))
        wall_h = time_hrt(rc, h, sets, inp, T, hs, 3, stream)
        rc.rc_cohort_run_chain(h, sets[0], step0_next(T), T, rc.RC_MODE_HOST_ROUNDTRIP, 0, C, stream)
        cnt = rc.rc_cohort_last_counts(h)
        us_h = wall_h / hs * 1e6
        out["host_roundtrip"] = {
            "value": round(trans_per_step / (us_h * 1e-6), 1), "unit": "transitions/s",
            "us_per_invocation": round(us_h, 3), "us_per_chained_step": round(us_h / T, 4),
            "host_over_resident": round(us_h / (ms_per_step * 1e3), 3),
            "launches_per_invocation": cnt[0], "d2h_copies_per_invocation": cnt[1], "steps": hs,
        }
        bits = floor_bits(rc, h, inp, T, stream)
        fcalls = Launches(rc, h, sets, T, [(0, C)], stream, bits)
        warm_calls(fcalls, None)
        wall_f = time_floor(rc, h, sets, bits, inp, T, args.steps, args.warmup, stream, calls=fcalls)
        us_f = wall_f / args.steps * 1e6
        out["floor"] = {
            "us_per_invocation": round(us_f, 3), "us_per_chained_step": round(us_f / T, 4),
            "resident_over_floor": round(ms_per_step * 1e3 / us_f, 3),
            "note": "no-decision floor: the resident chain replaying a recorded decision "
                    "bitmap with no predicate (a structural floor, not an online policy)",
        }
        if cpu is not None:
            if not args.no_kr:
                cpu["safe_suffix_k_r"] = safe_suffix_threshold(rc, wk)
            out["cpu_baseline"] = cpu
        out["hbm_measured"] = hbm_measured()
        props = torch.cuda.get_device_properties(0)
        out["device"] = {"name": props.name, "arch": getattr(props, "gcnArchName", None),
                         "compute_units": props.multi_processor_count,
                         "memory_GiB": round(props.total_memory / 2 ** 30, 1),
                         "l2_cache_MiB": round(getattr(props, "L2_cache_size", 0) / 2 ** 20, 1)}
        if not args.no_former:
            # launch-to-start budget: the measured synchronized invocation of
            # a 256-session, 16-step batch when the K_r sweep ran, else 25 us
            lat_us = 25.0
            kr = (cpu or {}).get("safe_suffix_k_r")
            if kr:
                lat_us = max(r["gpu_us"] for r in kr["rows"] if r["K"] == 256 and r["T"] == 16)
            out["cohort_former"] = cohort_former(rc, wk, int(round(lat_us * 1e3)))
        if not args.no_mechanisms:
            out["mechanisms"] = {k: mechanism_row(rc, wk, k, args.mech_rows, args.mech_row_ms * 1e-3,
                                                  args.mech_common_count) for k in wk.WORKLOAD_ORDER}
            out["mechanisms_paper_context"] = PAPER_CONTEXT
    rc.rc_cohort_destroy(h)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
