"""The oracle: a plain CPU implementation of the batched ready-cohort
control transition.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this package.  The product
path (``paper_2608_12123_amd``) never imports it and shares no code with it.

Two independent formulations live here:

* ``rc_oracle.c`` -- single-threaded C, built into ``librc_oracle.so`` and
  called through ctypes (:class:`Oracle`).  This is the parity reference for
  the GPU path.
* ``pyref.py`` -- the same definition written a second time with Python
  integers, used on tiny inputs to cross-check the C oracle.

The transition follows the paper's unit of work (Abstract; Section 2 "Unit of
execution"), its decision/route-body mechanism (Section 7 "Matched
mechanisms") and the per-event compaction and effect ordering it names as
missing (Section 11 "Mechanism and sampling scope").
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "rc_oracle.c")
LIB = os.path.join(HERE, "librc_oracle.so")

ROUTE_MOD = 0
ROUTE_CDF = 1


def build(force: bool = True, src: str = SRC, out: str = LIB) -> str:
    """Compile ``src`` (default ``rc_oracle.c``) with gcc into ``out``.

    Plain ``-O2``: no ``-march``, no vectorisation hints, no threads.
    """
    if not force and os.path.exists(out) and os.path.getmtime(out) >= os.path.getmtime(src):
        return out
    tmp = out + ".tmp%d" % os.getpid()
    cmd = ["gcc", "-std=c99", "-O2", "-fPIC", "-shared", "-Wall", "-Wextra",
           "-o", tmp, src]
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


def _p32(a):
    if a is None:
        return None
    assert a.dtype == np.uint32 and a.flags["C_CONTIGUOUS"], "need contiguous uint32"
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_uint32))


def _u32(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.uint32))


class Oracle:
    """ctypes view of one built oracle library."""

    def __init__(self, path: str = LIB):
        lib = ctypes.CDLL(path)
        u32 = ctypes.c_uint32
        p32 = ctypes.POINTER(ctypes.c_uint32)
        lib.rc_oracle_fmix32.argtypes = [u32]
        lib.rc_oracle_fmix32.restype = u32
        lib.rc_oracle_rotl.argtypes = [u32, u32]
        lib.rc_oracle_rotl.restype = u32
        lib.rc_oracle_route.argtypes = [u32, u32, u32, p32]
        lib.rc_oracle_route.restype = u32
        lib.rc_oracle_decide.argtypes = [u32, u32, u32, u32]
        lib.rc_oracle_decide.restype = u32
        lib.rc_oracle_update_word.argtypes = [u32, u32, u32, u32, u32, p32]
        lib.rc_oracle_update_word.restype = u32
        lib.rc_oracle_run_chain.argtypes = (
            [u32, u32, u32, u32, p32, p32, u32, p32, u32]
            + [p32] * 6 + [u32, u32, u32, u32, u32, p32])
        lib.rc_oracle_run_chain.restype = ctypes.c_int
        lib.rc_oracle_run_floor.argtypes = (
            [u32, u32, u32, u32, p32, p32, u32, p32, p32]
            + [p32] * 6 + [u32, u32, u32, u32])
        lib.rc_oracle_run_floor.restype = ctypes.c_int
        lib.rc_oracle_count_taken_all_outcomes.argtypes = [u32, u32, u32]
        lib.rc_oracle_count_taken_all_outcomes.restype = ctypes.c_uint64
        lib.rc_oracle_route_histogram.argtypes = [
            ctypes.c_uint64, ctypes.c_uint64, u32, u32, p32,
            ctypes.POINTER(ctypes.c_uint64)]
        lib.rc_oracle_route_histogram.restype = None
        self.lib = lib
        self.path = path

    def fmix32(self, h: int) -> int:
        return int(self.lib.rc_oracle_fmix32(h & 0xFFFFFFFF))

    def rotl(self, x: int, k: int) -> int:
        return int(self.lib.rc_oracle_rotl(x & 0xFFFFFFFF, k & 0xFFFFFFFF))

    def route(self, o: int, n_routes: int, route_mode: int, route_cdf=None) -> int:
        cdf = _u32(route_cdf) if route_cdf is not None else None
        return int(self.lib.rc_oracle_route(o & 0xFFFFFFFF, n_routes, route_mode, _p32(cdf)))

    def decide(self, s0: int, o: int, step: int, thr: int) -> int:
        return int(self.lib.rc_oracle_decide(s0 & 0xFFFFFFFF, o & 0xFFFFFFFF,
                                             step & 0xFFFFFFFF, thr))

    def update_word(self, x: int, w: int, r: int, d: int, o: int, table) -> int:
        t = _u32(table).ravel()
        return int(self.lib.rc_oracle_update_word(x & 0xFFFFFFFF, w, r, d,
                                                  o & 0xFFFFFFFF, _p32(t)))

    def count_taken_all_outcomes(self, s0: int, step: int, thr: int) -> int:
        return int(self.lib.rc_oracle_count_taken_all_outcomes(s0, step, thr))

    def route_histogram(self, lo: int, hi: int, n_routes: int, route_mode: int,
                        route_cdf=None) -> np.ndarray:
        counts = np.zeros(n_routes, dtype=np.uint64)
        cdf = _u32(route_cdf) if route_cdf is not None else None
        self.lib.rc_oracle_route_histogram(
            lo, hi, n_routes, route_mode, _p32(cdf),
            counts.ctypes.data_as(ctypes.POINTER(ctypes.c_uint64)))
        return counts

    def run_chain(self, *, n_words, n_routes, cohort_offsets, table, route_mode,
                  route_cdf, decide_thr, state, outcome, n_steps, step0=0,
                  cohort_begin=0, cohort_end=None, eff_sid=None, eff_tool=None,
                  eff_payload=None, n_taken=None, decisions=None, record=False):
        """Run ``n_steps`` chained steps in place.

        ``state`` is ``[W][ld]`` uint32 and ``outcome`` ``[ld]`` uint32; both
        are updated in place.  Effect arrays (``[T][ld]``, ``[T][ld]``,
        ``[T][ld][4]``) and ``n_taken`` (``[T][C]``) are allocated filled with
        ``0xFFFFFFFF`` when not given.  Returns a dict of the output arrays.

        ``decisions``: a ``[T][ceil(ld/32)]`` uint32 bitmap; when given, the
        no-decision floor runs instead (decisions read from it, no
        predicate).  ``record``: also return the decisions made, as such a
        bitmap (zero for sessions not stepped), under ``"decisions"``.
        """
        offsets = _u32(cohort_offsets)
        n_cohorts = offsets.size - 1
        n_sessions = int(offsets[-1])
        table = _u32(table).reshape(-1)
        cdf = _u32(route_cdf) if route_cdf is not None else None
        assert state.dtype == np.uint32 and outcome.dtype == np.uint32
        assert state.flags["C_CONTIGUOUS"] and outcome.flags["C_CONTIGUOUS"]
        ld = state.shape[1]
        assert state.shape[0] == n_words and outcome.shape[0] == ld
        T = n_steps
        if cohort_end is None:
            cohort_end = n_cohorts
        fill = np.uint32(0xFFFFFFFF)
        if eff_sid is None:
            eff_sid = np.full((T, ld), fill, dtype=np.uint32)
        if eff_tool is None:
            eff_tool = np.full((T, ld), fill, dtype=np.uint32)
        if eff_payload is None:
            eff_payload = np.full((T, ld, 4), fill, dtype=np.uint32)
        if n_taken is None:
            n_taken = np.full((T, n_cohorts), fill, dtype=np.uint32)
        dwords = (ld + 31) // 32
        if decisions is not None:
            bits = _u32(decisions)
            assert bits.shape == (T, dwords), "decisions must be [T][ceil(ld/32)]"
            rc = self.lib.rc_oracle_run_floor(
                n_sessions, n_words, n_routes, n_cohorts, _p32(offsets), _p32(table),
                route_mode, _p32(cdf), _p32(bits), _p32(state), _p32(outcome),
                _p32(eff_sid), _p32(eff_tool), _p32(eff_payload), _p32(n_taken),
                ld, T, cohort_begin, cohort_end)
            if rc != 0:
                raise ValueError("rc_oracle_run_floor returned %d" % rc)
            rec = None
        else:
            rec = np.zeros((T, dwords), dtype=np.uint32) if record else None
            rc = self.lib.rc_oracle_run_chain(
                n_sessions, n_words, n_routes, n_cohorts, _p32(offsets), _p32(table),
                route_mode, _p32(cdf), decide_thr, _p32(state), _p32(outcome),
                _p32(eff_sid), _p32(eff_tool), _p32(eff_payload), _p32(n_taken),
                ld, step0 & 0xFFFFFFFF, T, cohort_begin, cohort_end, _p32(rec))
            if rc != 0:
                raise ValueError("rc_oracle_run_chain returned %d" % rc)
        out = {"state": state, "outcome": outcome, "eff_sid": eff_sid,
               "eff_tool": eff_tool, "eff_payload": eff_payload, "n_taken": n_taken}
        if rec is not None:
            out["decisions"] = rec
        return out

    def run_inputs(self, inp, n_steps=None, step0=0, cohort_begin=0, cohort_end=None,
                   decisions=None, record=False):
        """Run on a copy of an input bundle from the workload generator."""
        state, outcome = inp.state.copy(), inp.outcome.copy()
        return self.run_chain(
            n_words=inp.n_words, n_routes=inp.n_routes,
            cohort_offsets=inp.cohort_offsets, table=inp.table,
            route_mode=inp.route_mode, route_cdf=inp.route_cdf,
            decide_thr=inp.decide_thr, state=state, outcome=outcome,
            n_steps=inp.n_steps if n_steps is None else n_steps, step0=step0,
            cohort_begin=cohort_begin, cohort_end=cohort_end, decisions=decisions,
            record=record)


_default = None


def load() -> Oracle:
    """The built oracle library (built only if it is absent)."""
    global _default
    if _default is None:
        if not os.path.exists(LIB):
            build()
        _default = Oracle(LIB)
    return _default
