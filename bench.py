"""Benchmark of the batched ready-cohort transition on one MI355X.

Default run (no flags): the 100,000-session workload (391 cohorts of K=256,
W=32, R=256, p=0.5, T=16 chained steps) -- the throughput / HBM-bandwidth
workload.  One bench step is one device-resident chain over all sessions
(every step of the hot path: route, decide, compact, update, emit, chain).
It prints ONE JSON line with the contract fields plus:

* ``roofline``: algorithmic bytes per launch of the resident chain kernel
  over its average duration, timed with HIP events on the launch stream,
  with the HBM traffic of the committed rocprofv3 counter summary;
* ``valu``: VALU instructions per launch (committed SQ counter summary) and
  the fraction of the chip's VALU issue they occupy;
* ``host_roundtrip``: the same workload through the host-round-trip
  mechanism (4-byte readback + host branch + relaunch every chained step);
* ``floor``: the no-decision floor (decisions replayed from a bitmap);
* ``mechanisms``: resident, synchronized resident, floor and host round trip
  on all five workloads (median of timed rows: microseconds per invocation
  and per chained step, launches and device-to-host copies per invocation);
* ``cpu_baseline``: the single-threaded CPU oracle on the same workload, and
  the safe-suffix threshold K_r (batch sizes and chain lengths where the
  resident chain beats the oracle on one core and on all cores);
* ``cohort_former``: the cohort shares F, P*, U, the online share A and
  their ratios on seeded 1M-event arrival streams;
* ``hbm_measured`` and ``device``: measured copy and fill bandwidth and the
  device's properties, beside the spec peak.

Inputs are synthetic and seeded (see paper_2608_12123_amd/workload.py).  The
timed region rotates through enough buffer sets that the working set is
larger than the 256 MB Infinity Cache.
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


def time_resident(rc, h, sets, inp, T, steps, warmup, stream, ranges=None):
    """Pipelined resident chains.  Returns the wall seconds of the timed loop
    and its GPU time (ms) from one HIP event pair around it, recorded on the
    stream the kernels are launched on (the current torch stream, whose
    handle is passed to the library).  Nothing else is enqueued between the
    launches, so region time / steps is the average launch duration plus the
    small gap between back-to-back launches."""
    import torch
    C = inp.n_cohorts
    rng = ranges or [(0, C)]
    cur = torch.cuda.current_stream()
    assert cur.cuda_stream == stream
    for i in range(warmup):
        cb, ce = rng[i % len(rng)]
        rc.rc_cohort_run_chain(h, sets[i], 0, T, rc.RC_MODE_RESIDENT, cb, ce, stream)
    r0, r1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    r0.record(cur)
    for i in range(steps):
        cb, ce = rng[i % len(rng)]
        rc.rc_cohort_run_chain(h, sets[i], 0, T, rc.RC_MODE_RESIDENT, cb, ce, stream)
    r1.record(cur)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    return wall, r0.elapsed_time(r1)


def time_resident_synced(rc, h, sets, inp, T, steps, stream, ranges):
    import torch
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(steps):
        cb, ce = ranges[i % len(ranges)]
        rc.rc_cohort_run_chain(h, sets[i], 0, T, rc.RC_MODE_RESIDENT, cb, ce, stream)
        torch.cuda.current_stream().synchronize()
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


def time_floor(rc, h, sets, bits, inp, T, steps, warmup, stream, ranges=None):
    """Pipelined no-decision-floor launches (same protocol as the resident
    chain).  Returns the wall seconds of the timed loop."""
    import torch
    rng = ranges or [(0, inp.n_cohorts)]
    ptr = bits.data_ptr()
    for i in range(warmup):
        cb, ce = rng[i % len(rng)]
        rc.rc_cohort_run_floor(h, sets[i], ptr, T, cb, ce, stream)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(steps):
        cb, ce = rng[i % len(rng)]
        rc.rc_cohort_run_floor(h, sets[i], ptr, T, cb, ce, stream)
    torch.cuda.synchronize()
    return time.perf_counter() - t0


def time_hrt(rc, h, sets, inp, T, steps, warmup, stream, ranges=None):
    import torch
    C = inp.n_cohorts
    rng = ranges or [(0, C)]
    for i in range(warmup):
        cb, ce = rng[i % len(rng)]
        rc.rc_cohort_run_chain(h, sets[i], 0, T, rc.RC_MODE_HOST_ROUNDTRIP, cb, ce, stream)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(steps):
        cb, ce = rng[i % len(rng)]
        rc.rc_cohort_run_chain(h, sets[i], 0, T, rc.RC_MODE_HOST_ROUNDTRIP, cb, ce, stream)
    torch.cuda.synchronize()
    return time.perf_counter() - t0


MECH_ROWS = 9  # timed rows per mechanism and workload (median reported)


def _rows(timed, n_per_row, rows=MECH_ROWS):
    """Microseconds per invocation of `rows` timed rows of n_per_row
    invocations each: (median, 10th percentile, 90th percentile)."""
    us = [timed(n_per_row) / n_per_row * 1e6 for _ in range(rows)]
    return float(np.median(us)), float(np.percentile(us, 10)), float(np.percentile(us, 90))


def mechanism_row(rc, wk, key, budget_s=1.0):
    """Resident (pipelined and synchronized), no-decision floor and host
    round trip on one workload, invocations as the workload defines them.
    Protocol: warmups, a calibration of the invocation count on the faster
    (resident) mechanism, then MECH_ROWS timed rows per mechanism; the
    median row is reported with its 10th-90th percentile spread."""
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
        else:
            ranges = [(0, inp.n_cohorts)]
            per_inv = inp.n_sessions * T
        sets = Sets(rc, inp, T, 1 if wl.per_cohort_invocation else 2)
        stream = torch.cuda.current_stream().cuda_stream
        # warm up, then calibrate the invocations per row on the resident mechanism
        w, _ = time_resident(rc, h, sets, inp, T, 20, 5, stream, ranges)
        n = int(max(10, min(20000, budget_s / 4 / MECH_ROWS / max(w / 20, 1e-7))))
        r_med, r_lo, r_hi = _rows(lambda k: time_resident(rc, h, sets, inp, T, k, 0, stream, ranges)[0], n)
        rc.rc_cohort_run_chain(h, sets[0], 0, T, rc.RC_MODE_RESIDENT, *ranges[0], stream)
        res_counts = rc.rc_cohort_last_counts(h)
        n_sync = max(5, n // 4)
        s_med, s_lo, s_hi = _rows(lambda k: time_resident_synced(rc, h, sets, inp, T, k, stream, ranges),
                                  n_sync)
        bits = floor_bits(rc, h, inp, T, stream)
        time_floor(rc, h, sets, bits, inp, T, 5, 5, stream, ranges)
        f_med, f_lo, f_hi = _rows(lambda k: time_floor(rc, h, sets, bits, inp, T, k, 0, stream, ranges), n)
        w1 = time_hrt(rc, h, sets, inp, T, 3, 1, stream, ranges)
        n_h = int(max(3, min(n, budget_s / 4 / MECH_ROWS / max(w1 / 3, 1e-7))))
        h_med, h_lo, h_hi = _rows(lambda k: time_hrt(rc, h, sets, inp, T, k, 0, stream, ranges), n_h)
        rc.rc_cohort_run_chain(h, sets[0], 0, T, rc.RC_MODE_HOST_ROUNDTRIP, *ranges[0], stream)
        hrt_counts = rc.rc_cohort_last_counts(h)
        torch.cuda.synchronize()
    finally:
        rc.rc_cohort_destroy(h)
    spread = lambda lo, hi: [round(lo, 3), round(hi, 3)]
    return {
        "workload": wl.title, "T": T, "transitions_per_invocation": per_inv,
        "resident_us_per_invocation": round(r_med, 3),
        "resident_us_p10_p90": spread(r_lo, r_hi),
        "resident_us_per_chained_step": round(r_med / T, 4),
        "resident_synced_us_per_invocation": round(s_med, 3),
        "resident_synced_us_p10_p90": spread(s_lo, s_hi),
        "host_rt_us_per_invocation": round(h_med, 3),
        "host_rt_us_p10_p90": spread(h_lo, h_hi),
        "host_rt_us_per_chained_step": round(h_med / T, 4),
        "host_over_resident": round(h_med / r_med, 3),
        "host_over_resident_synced": round(h_med / s_med, 3),
        "floor_us_per_invocation": round(f_med, 3),
        "floor_us_p10_p90": spread(f_lo, f_hi),
        "resident_over_floor": round(r_med / f_med, 3),
        "resident_transitions_per_s": round(per_inv / (r_med * 1e-6), 1),
        "host_rt_transitions_per_s": round(per_inv / (h_med * 1e-6), 1),
        "launches_per_invocation": {"resident": res_counts[0], "host_rt": hrt_counts[0]},
        "d2h_copies_per_invocation": {"resident": res_counts[1], "host_rt": hrt_counts[1]},
        "invocations_per_row": {"resident": n, "resident_synced": n_sync, "host_rt": n_h, "floor": n},
        "rows": MECH_ROWS,
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
                      % (inp.n_sessions, T, reps, el, platform.processor() or platform.machine(),
                         os.cpu_count() or 0)}, first


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
    args = ap.parse_args()

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

    wall, region_ms = time_resident(rc, h, sets, inp, T, args.steps, args.warmup, stream)
    trans_per_step = N * T
    value = trans_per_step * args.steps / wall
    ms_per_step = wall / args.steps * 1e3
    k_avg_ms = region_ms / args.steps
    abytes = algorithmic_bytes(N, W, T, C)
    achieved = abytes / (k_avg_ms * 1e-3) / 1e9
    traffic = stored_traffic(wl.key)
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
                                "loop, divided by the launches"},
        "roofline": {
            "bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4),
            "traffic": traffic,
            "kernel": "rc_chain_kernel", "algorithmic_bytes_per_launch": abytes,
        },
        "verified_vs_oracle": verified,
    }
    valu = stored_valu(wl.key)
    if valu is not None:
        cus = torch.cuda.get_device_properties(0).multi_processor_count
        busy = valu["insts_per_launch"] * 4.0 / (4 * cus * ENGINE_CLOCK_HZ * k_avg_ms * 1e-3)
        out["valu"] = {"insts_per_launch": valu["insts_per_launch"],
                       "insts_per_wave": round(valu["insts_per_launch"] / valu["waves"], 1),
                       "busy_frac": round(busy, 4),
                       "basis": "SQ_INSTS_VALU (committed rocprofv3 summary) x 4 cycles / "
                                "(4 SIMDs x CUs x 2.4 GHz x measured kernel time)"}
    if not args.profile_only:
        hs = max(5, min(args.hrt_steps, args.steps))
        wall_h = time_hrt(rc, h, sets, inp, T, hs, 3, stream)
        rc.rc_cohort_run_chain(h, sets[0], 0, T, rc.RC_MODE_HOST_ROUNDTRIP, 0, C, stream)
        cnt = rc.rc_cohort_last_counts(h)
        us_h = wall_h / hs * 1e6
        out["host_roundtrip"] = {
            "value": round(trans_per_step / (us_h * 1e-6), 1), "unit": "transitions/s",
            "us_per_invocation": round(us_h, 3), "us_per_chained_step": round(us_h / T, 4),
            "host_over_resident": round(us_h / (ms_per_step * 1e3), 3),
            "launches_per_invocation": cnt[0], "d2h_copies_per_invocation": cnt[1], "steps": hs,
        }
        bits = floor_bits(rc, h, inp, T, stream)
        wall_f = time_floor(rc, h, sets, bits, inp, T, args.steps, args.warmup, stream)
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
            out["mechanisms"] = {k: mechanism_row(rc, wk, k) for k in wk.WORKLOAD_ORDER}
    rc.rc_cohort_destroy(h)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
