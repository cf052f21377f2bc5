"""Streams and concurrent handles (needs an MI355X).

Every call takes a raw hipStream_t and orders its work on that stream: the
inputs are written by asynchronous copies queued on a side stream behind
slow work, and the outputs are read back by asynchronous copies queued on
the same stream right after the call.  If the library launched anywhere
else, it would read the inputs before they are written or be read before it
finishes.  Two handles of different shapes (split full image, table image)
run at once on two streams from two host threads, in both mechanisms; each
result equals the oracle's bit for bit.
"""
import sys
import threading

import numpy as np
import pytest

import oracle
from paper_2608_12123_amd import rc_cohort as rc
from paper_2608_12123_amd import workload as wk

pytestmark = pytest.mark.gpu

KEYS = ("state", "outcome", "eff_sid", "eff_tool", "eff_payload", "n_taken")

# (W, R, route mode, thr, cohort sizes, T, step0)
CASES = [
    (32, 256, wk.ROUTE_MOD, 32768, [256] * 40 + [160], 16, 5),
    (64, 1024, wk.ROUTE_CDF, 3277, [256, 31, 32, 100, 1, 64, 200, 128, 77] * 5, 8, 0xFFFFFFFC),
]


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def orc():
    oracle.build(force=False)
    return oracle.load()


def pinned(arr: np.ndarray):
    import torch
    t = torch.from_numpy(np.ascontiguousarray(arr).view(np.int32))
    return t.pin_memory()


def on_stream(co, state, outcome, stream, step0, T, mode, busy, out):
    """Queue slow work, the input copies, the chain and the output copies on
    ``stream``; wait for the stream only at the end."""
    import torch
    try:
        with torch.cuda.stream(stream):
            for _ in range(8):
                busy.add_(1)
            co.t["state"].copy_(state, non_blocking=True)
            co.t["outcome"].copy_(outcome, non_blocking=True)
            co.run_chain(step0, T, mode, stream=stream.cuda_stream)
            host = {}
            for k in KEYS:
                src = co.t[k] if k in ("state", "outcome") else co.t[k][:T]
                host[k] = torch.empty(src.shape, dtype=torch.int32, pin_memory=True)
                host[k].copy_(src, non_blocking=True)
        stream.synchronize()
        out["got"] = {k: v.numpy().view(np.uint32).copy() for k, v in host.items()}
    except BaseException as e:  # reported by the main thread
        out["error"] = e


@pytest.mark.parametrize("mode", ["resident", "host round trip"])
def test_two_handles_two_streams_two_threads(orc, mode):
    import torch
    m = rc.RC_MODE_RESIDENT if mode == "resident" else rc.RC_MODE_HOST_ROUNDTRIP
    jobs = []
    for i, (W, R, rmode, thr, sizes, T, step0) in enumerate(CASES):
        inp = wk.make_custom(n_words=W, n_routes=R, route_mode=rmode, decide_thr=thr,
                             cohort_sizes=sizes, n_steps=T, seed_key=33_000 + i,
                             ld=sum(sizes) + 32)
        say("streams %s: handle %d W=%d R=%d C=%d N=%d T=%d" % (mode, i, W, R, inp.n_cohorts,
                                                             inp.n_sessions, T))
        want = orc.run_inputs(inp, n_steps=T, step0=step0)
        co = rc.Cohort(n_words=W, n_routes=R, cohort_offsets=inp.cohort_offsets,
                       table=inp.table, route_mode=rmode, route_cdf=inp.route_cdf,
                       decide_thr=thr, max_steps=T, ld=inp.ld)
        busy = torch.zeros(64 << 20, dtype=torch.int32, device=co.device)
        jobs.append(dict(co=co, want=want, state=pinned(inp.state), outcome=pinned(inp.outcome),
                         stream=torch.cuda.Stream(device=co.device), step0=step0, T=T,
                         busy=busy, out={}))
    torch.cuda.synchronize()  # buffers were filled on the default stream
    try:
        threads = [threading.Thread(target=on_stream,
                                    args=(j["co"], j["state"], j["outcome"], j["stream"],
                                          j["step0"], j["T"], m, j["busy"], j["out"]))
                   for j in jobs]
        for t in threads:
            t.start()
        for t in threads:
            t.join(timeout=100)
            assert not t.is_alive(), "a stream did not finish"
        for i, j in enumerate(jobs):
            if "error" in j["out"]:
                raise j["out"]["error"]
            got, want = j["out"]["got"], j["want"]
            for k in KEYS:
                assert np.array_equal(got[k], want[k]), (mode, i, k)
    finally:
        torch.cuda.synchronize()
        for j in jobs:
            j["co"].close()


def advanced(b: "rc.RcBuffers", ld: int, t: int, n_cohorts: int) -> "rc.RcBuffers":
    """The buffers of b with the effect log and counts advanced by t slices
    (the pointers a caller passes to continue a chain in the same log)."""
    return rc.RcBuffers(b.state, b.outcome, b.eff_sid + 4 * t * ld, b.eff_tool + 4 * t * ld,
                        b.eff_payload + 16 * t * ld, b.n_taken + 4 * t * n_cohorts, ld)


def one_handle_two_streams(orc, entry):
    """A chain continued on another stream by the same handle, with no
    synchronization by the caller: the second host-round-trip call must wait
    for the first call's last body kernels (its scratch and the state they
    write), so the two calls equal one chain of T1 + T2 steps."""
    import torch
    W, R, thr, T1, T2 = 32, 64, 19661, 5, 4
    sizes = [256] * 30 + [100, 64, 17]
    inp = wk.make_custom(n_words=W, n_routes=R, route_mode=wk.ROUTE_CDF, decide_thr=thr,
                         cohort_sizes=sizes, n_steps=T1 + T2, seed_key=33_100, ld=sum(sizes) + 64)
    say("one handle, two streams (%s): N=%d T=%d+%d" % (entry, inp.n_sessions, T1, T2))
    want = orc.run_inputs(inp, n_steps=T1 + T2)
    co = rc.Cohort.from_inputs(inp, max_steps=T1 + T2)
    fn = getattr(rc, "rc_cohort_" + entry)
    try:
        torch.cuda.synchronize()
        sa, sb = torch.cuda.Stream(device=co.device), torch.cuda.Stream(device=co.device)
        for rep in range(3):
            co.upload(inp.state, inp.outcome)
            torch.cuda.synchronize()
            fn(co.handle, co.buffers, 0, T1, rc.RC_MODE_HOST_ROUNDTRIP, 0, co.n_cohorts,
               sa.cuda_stream)
            fn(co.handle, advanced(co.buffers, co.ld, T1, co.n_cohorts), T1, T2,
               rc.RC_MODE_HOST_ROUNDTRIP, 0, co.n_cohorts, sb.cuda_stream)
            sb.synchronize()
            got = co.download(T1 + T2)
            for k in KEYS:
                assert np.array_equal(got[k], want[k]), (entry, rep, k)
    finally:
        torch.cuda.synchronize()
        co.close()


def test_one_handle_host_round_trip_on_two_streams(orc):
    one_handle_two_streams(orc, "run_chain")
