"""Thin Python binding of ``librc_cohort.so`` (the C ABI in include/rc_cohort.h).

Argument marshalling only: every step of the transition runs in the HIP
kernels.  There is no CPU fallback -- if the library is missing or no gfx950
device is usable, the calls raise.

The function names are those of the C ABI (``rc_cohort_create``,
``rc_cohort_step``, ``rc_cohort_run_chain``, ``rc_cohort_destroy``, ...).
Device buffers are torch int32 tensors (PyTorch supplies device memory and
streams); uint32 values are carried bit-for-bit in int32 storage.
"""
from __future__ import annotations

import ctypes
import os
from typing import Dict, Optional

import numpy as np

PKG = os.path.dirname(os.path.abspath(__file__))
# RC_COHORT_LIB names another build of the same sources, e.g. the host-only
# sanitizer build of the CPU tests (which holds no GPU entry point).
LIB_PATH = os.environ.get("RC_COHORT_LIB") or os.path.join(PKG, "librc_cohort.so")

RC_OK, RC_E_INVALID, RC_E_NOMEM, RC_E_DEVICE = 0, 1, 2, 3
RC_ROUTE_MOD, RC_ROUTE_CDF = 0, 1
RC_MODE_RESIDENT, RC_MODE_HOST_ROUNDTRIP = 0, 1
# Shape limits of a descriptor (the #defines of rc_cohort.h).
RC_MIN_WORDS, RC_MAX_WORDS = 4, 64
RC_MAX_ROUTES = 1024
RC_MAX_COHORT = 256
RC_MAX_SESSIONS = 1 << 28
RC_NOALLOC_MAX_SESSIONS = 1 << 20

EXPORTED = [
    "rc_cohort_create", "rc_cohort_step", "rc_cohort_run_chain", "rc_cohort_run_floor",
    "rc_cohort_run_chain_noalloc",
    "rc_cohort_destroy", "rc_status_string", "rc_cohort_last_counts", "rc_cohort_plan_info",
    "rc_plan_lanes", "rc_pack_shares", "rc_online_compact", "rc_cohorts_from_batches",
]
# entry points that need no device (the host-only build holds only these)
HOST_ONLY = ["rc_status_string", "rc_plan_lanes", "rc_pack_shares", "rc_online_compact",
             "rc_cohorts_from_batches"]

_P32 = ctypes.POINTER(ctypes.c_uint32)


class RcCohortDesc(ctypes.Structure):
    _fields_ = [
        ("n_sessions", ctypes.c_uint32),
        ("n_words", ctypes.c_uint32),
        ("n_routes", ctypes.c_uint32),
        ("n_cohorts", ctypes.c_uint32),
        ("cohort_offsets", _P32),
        ("table", _P32),
        ("route_mode", ctypes.c_uint32),
        ("route_cdf", _P32),
        ("decide_thr", ctypes.c_uint32),
    ]


class RcBuffers(ctypes.Structure):
    _fields_ = [
        ("state", ctypes.c_void_p),
        ("outcome", ctypes.c_void_p),
        ("eff_sid", ctypes.c_void_p),
        ("eff_tool", ctypes.c_void_p),
        ("eff_payload", ctypes.c_void_p),
        ("n_taken", ctypes.c_void_p),
        ("ld", ctypes.c_uint32),
    ]


class RcPackResult(ctypes.Structure):
    _fields_ = [
        ("n_events", ctypes.c_uint64),
        ("fixed_eligible", ctypes.c_uint64),
        ("packed", ctypes.c_uint64),
        ("overlap_eligible", ctypes.c_uint64),
        ("n_batches", ctypes.c_uint64),
    ]


class RcOnlineResult(ctypes.Structure):
    _fields_ = [
        ("n_events", ctypes.c_uint64),
        ("accelerated", ctypes.c_uint64),
        ("fallback_deadline", ctypes.c_uint64),
        ("fallback_capacity", ctypes.c_uint64),
        ("n_batches", ctypes.c_uint64),
        ("launched_at_capacity", ctypes.c_uint64),
    ]


class RcError(RuntimeError):
    def __init__(self, status: int, what: str):
        self.status = status
        super().__init__("%s failed: %s" % (what, rc_status_string(status)))


_lib: Optional[ctypes.CDLL] = None


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load the built HIP library.  Raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(
            "librc_cohort.so is not built (run paper_2608_12123_amd/build.py or "
            "__graft_entry__.build()); there is no CPU fallback")
    lib = ctypes.CDLL(path)
    missing = [n for n in EXPORTED if not hasattr(lib, n)]
    if missing and (path == os.path.join(PKG, "librc_cohort.so") or set(missing) & set(HOST_ONLY)):
        raise RuntimeError("%s lacks %s" % (path, ", ".join(missing)))
    _declare_host(lib)
    if "rc_cohort_create" in missing:
        # a host-only build (no device entry point)
        _lib = lib
        return lib
    lib.rc_cohort_create.argtypes = [ctypes.POINTER(RcCohortDesc), ctypes.c_int,
                                     ctypes.POINTER(ctypes.c_void_p)]
    lib.rc_cohort_create.restype = ctypes.c_int
    lib.rc_cohort_step.argtypes = [ctypes.c_void_p, ctypes.POINTER(RcBuffers), ctypes.c_uint32,
                                   ctypes.c_uint32, ctypes.c_uint32, ctypes.c_void_p]
    lib.rc_cohort_step.restype = ctypes.c_int
    lib.rc_cohort_run_chain.argtypes = [ctypes.c_void_p, ctypes.POINTER(RcBuffers), ctypes.c_uint32,
                                        ctypes.c_uint32, ctypes.c_int, ctypes.c_uint32,
                                        ctypes.c_uint32, ctypes.c_void_p]
    lib.rc_cohort_run_chain.restype = ctypes.c_int
    lib.rc_cohort_run_floor.argtypes = [ctypes.c_void_p, ctypes.POINTER(RcBuffers), ctypes.c_void_p,
                                        ctypes.c_uint32, ctypes.c_uint32, ctypes.c_uint32,
                                        ctypes.c_void_p]
    lib.rc_cohort_run_floor.restype = ctypes.c_int
    if "rc_cohort_run_chain_noalloc" not in missing:
        lib.rc_cohort_run_chain_noalloc.argtypes = lib.rc_cohort_run_chain.argtypes
        lib.rc_cohort_run_chain_noalloc.restype = ctypes.c_int
    lib.rc_cohort_destroy.argtypes = [ctypes.c_void_p]
    lib.rc_cohort_destroy.restype = ctypes.c_int
    lib.rc_cohort_last_counts.argtypes = [ctypes.c_void_p, _P32, _P32]
    lib.rc_cohort_last_counts.restype = ctypes.c_int
    lib.rc_cohort_plan_info.argtypes = [ctypes.c_void_p, _P32, _P32, _P32]
    lib.rc_cohort_plan_info.restype = ctypes.c_int
    _lib = lib
    return lib


def _declare_host(lib: ctypes.CDLL):
    lib.rc_status_string.argtypes = [ctypes.c_int]
    lib.rc_status_string.restype = ctypes.c_char_p
    lib.rc_plan_lanes.argtypes = [ctypes.POINTER(RcCohortDesc), ctypes.c_uint32, _P32, _P32,
                                  ctypes.c_uint32, _P32]
    lib.rc_plan_lanes.restype = ctypes.c_int
    lib.rc_pack_shares.argtypes = [ctypes.POINTER(ctypes.c_int64), _P32, ctypes.c_uint64, _P32,
                                   ctypes.c_uint32, ctypes.c_int64, ctypes.c_int64, _P32,
                                   ctypes.POINTER(RcPackResult)]
    lib.rc_pack_shares.restype = ctypes.c_int
    lib.rc_online_compact.argtypes = [ctypes.POINTER(ctypes.c_int64), _P32, ctypes.c_uint64, _P32,
                                      ctypes.c_uint32, ctypes.c_int64, ctypes.c_int64,
                                      ctypes.c_uint32, _P32, ctypes.POINTER(ctypes.c_int64),
                                      ctypes.POINTER(RcOnlineResult)]
    lib.rc_online_compact.restype = ctypes.c_int
    lib.rc_cohorts_from_batches.argtypes = [_P32, ctypes.c_uint64, ctypes.c_uint64, ctypes.c_uint32,
                                            _P32, _P32, ctypes.POINTER(ctypes.c_uint64)]
    lib.rc_cohorts_from_batches.restype = ctypes.c_int


def _u32(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.uint32))


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(_P32)


def _stream_handle(stream) -> Optional[int]:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def rc_status_string(status: int) -> str:
    return load_library().rc_status_string(status).decode()


def _check(status: int, what: str):
    if status != RC_OK:
        raise RcError(status, what)


def rc_cohort_create(*, n_sessions: int, n_words: int, n_routes: int, cohort_offsets,
                     table, route_mode: int, route_cdf, decide_thr: int, device: int = 0,
                     check: bool = True):
    """Create a handle; returns (status, handle) when ``check`` is False."""
    lib = load_library()
    off = _u32(cohort_offsets)
    tab = _u32(table).reshape(-1)
    cdf = None if route_cdf is None else _u32(route_cdf)
    desc = RcCohortDesc(n_sessions, n_words, n_routes, off.size - 1, _ptr(off), _ptr(tab),
                        route_mode, _ptr(cdf), decide_thr)
    h = ctypes.c_void_p()
    st = lib.rc_cohort_create(ctypes.byref(desc), device, ctypes.byref(h))
    if not check:
        return st, h
    _check(st, "rc_cohort_create")
    return h


def rc_cohort_step(h, buffers: RcBuffers, step: int, cohort_begin: int, cohort_end: int,
                   stream=None, check: bool = True) -> int:
    st = load_library().rc_cohort_step(h, ctypes.byref(buffers), step & 0xFFFFFFFF,
                                       cohort_begin, cohort_end, _stream_handle(stream))
    if check:
        _check(st, "rc_cohort_step")
    return st


def rc_cohort_run_chain(h, buffers: RcBuffers, step0: int, n_steps: int, mode: int,
                        cohort_begin: int, cohort_end: int, stream=None,
                        check: bool = True) -> int:
    st = load_library().rc_cohort_run_chain(h, ctypes.byref(buffers), step0 & 0xFFFFFFFF,
                                            n_steps, mode, cohort_begin, cohort_end,
                                            _stream_handle(stream))
    if check:
        _check(st, "rc_cohort_run_chain")
    return st


def rc_cohort_run_chain_noalloc(h, buffers: RcBuffers, step0: int, n_steps: int, mode: int,
                                cohort_begin: int, cohort_end: int, stream=None,
                                check: bool = True) -> int:
    """rc_cohort_run_chain with the host round trip's scratch in the
    library's fixed device array (no device allocation by the call)."""
    st = load_library().rc_cohort_run_chain_noalloc(h, ctypes.byref(buffers), step0 & 0xFFFFFFFF,
                                                    n_steps, mode, cohort_begin, cohort_end,
                                                    _stream_handle(stream))
    if check:
        _check(st, "rc_cohort_run_chain_noalloc")
    return st


def rc_cohort_run_floor(h, buffers: RcBuffers, decisions_ptr: int, n_steps: int,
                        cohort_begin: int, cohort_end: int, stream=None, check: bool = True) -> int:
    """The no-decision floor; ``decisions_ptr`` is the device address of a
    ``[n_steps][ceil(ld/32)]`` uint32 decision bitmap."""
    st = load_library().rc_cohort_run_floor(h, ctypes.byref(buffers), decisions_ptr, n_steps,
                                            cohort_begin, cohort_end, _stream_handle(stream))
    if check:
        _check(st, "rc_cohort_run_floor")
    return st


def rc_cohort_destroy(h) -> int:
    return load_library().rc_cohort_destroy(h)


def rc_cohort_last_counts(h):
    a, b = ctypes.c_uint32(), ctypes.c_uint32()
    _check(load_library().rc_cohort_last_counts(h, ctypes.byref(a), ctypes.byref(b)),
           "rc_cohort_last_counts")
    return a.value, b.value


def rc_cohort_plan_info(h):
    a, b, c = ctypes.c_uint32(), ctypes.c_uint32(), ctypes.c_uint32()
    _check(load_library().rc_cohort_plan_info(h, ctypes.byref(a), ctypes.byref(b), ctypes.byref(c)),
           "rc_cohort_plan_info")
    return a.value, b.value, c.value


def rc_plan_lanes(*, cohort_offsets, n_words=4, n_routes=1, lanes_per_workgroup=256):
    """Host-only plan inspection: (lane_session, lane_cohort) uint32 arrays,
    one entry per plan lane, 0xFFFFFFFF for idle lanes."""
    lib = load_library()
    off = _u32(cohort_offsets)
    tab = np.zeros(n_routes * 16, dtype=np.uint32)
    desc = RcCohortDesc(int(off[-1]), n_words, n_routes, off.size - 1, _ptr(off), _ptr(tab),
                        RC_ROUTE_MOD, None, 32768)
    n = ctypes.c_uint32()
    _check(lib.rc_plan_lanes(ctypes.byref(desc), lanes_per_workgroup, None, None, 0,
                             ctypes.byref(n)), "rc_plan_lanes")
    ses = np.empty(n.value, dtype=np.uint32)
    coh = np.empty(n.value, dtype=np.uint32)
    _check(lib.rc_plan_lanes(ctypes.byref(desc), lanes_per_workgroup, _ptr(ses), _ptr(coh),
                             n.value, ctypes.byref(n)), "rc_plan_lanes")
    return ses, coh


def rc_pack_shares(*, release_ns, route, k_of_route, delta_ns: int, window_origin_ns: int = 0,
                   witness: bool = False, check: bool = True):
    """Cohort shares (numerators of F, P*, U) of a set of events; with
    ``witness``, also the batch of every event (0xFFFFFFFF: left out).
    Host computation in the library (no device)."""
    t = np.ascontiguousarray(release_ns, dtype=np.int64)
    r = _u32(route)
    k = _u32(k_of_route)
    n = t.size
    assert r.size == n
    bat = np.empty(n, dtype=np.uint32) if witness else None
    res = RcPackResult()
    st = load_library().rc_pack_shares(
        t.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)) if n else None, _ptr(r) if n else None,
        n, _ptr(k), k.size, int(delta_ns), int(window_origin_ns),
        _ptr(bat) if witness and n else None, ctypes.byref(res))
    if check:
        _check(st, "rc_pack_shares")
    if st != RC_OK:
        return st
    out = {"n_events": res.n_events, "fixed_eligible": res.fixed_eligible, "packed": res.packed,
           "overlap_eligible": res.overlap_eligible, "n_batches": res.n_batches}
    return (out, bat) if witness else out


UNLIMITED = 0xFFFFFFFF  # queue capacity without a limit


def _p64(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(ctypes.POINTER(ctypes.c_int64))


def rc_online_compact(*, release_ns, route, k_of_route, delta_ns: int, latency_ns: int = 0,
                      capacity: int = UNLIMITED, witness: bool = False, check: bool = True):
    """The online route compactor's counts (A's numerator and the
    fallbacks); with ``witness``, also the batch of every event
    (0xFFFFFFFF: CPU) and every batch's launch time.  Host computation in
    the library (no device)."""
    t = np.ascontiguousarray(release_ns, dtype=np.int64)
    r = _u32(route)
    k = _u32(k_of_route)
    n = t.size
    assert r.size == n
    bat = np.empty(n, dtype=np.uint32) if witness else None
    lt = np.empty(max(n, 1), dtype=np.int64) if witness else None
    res = RcOnlineResult()
    st = load_library().rc_online_compact(
        _p64(t) if n else None, _ptr(r) if n else None, n, _ptr(k), k.size, int(delta_ns),
        int(latency_ns), int(capacity), _ptr(bat) if witness and n else None,
        _p64(lt) if witness else None, ctypes.byref(res))
    if check:
        _check(st, "rc_online_compact")
    if st != RC_OK:
        return st
    out = {f: getattr(res, f) for f, _ in RcOnlineResult._fields_}
    return (out, bat, lt[:res.n_batches].copy()) if witness else out


def rc_cohorts_from_batches(batch_of_event, n_batches: int, max_cohort: int = 256,
                            check: bool = True):
    """(order, offsets): sessions grouped by cohort (event indices) and the
    cohort offsets, each batch cut into near-equal cohorts of at most
    ``max_cohort``."""
    b = _u32(batch_of_event)
    n = b.size
    order = np.empty(max(n, 1), dtype=np.uint32)
    offsets = np.empty(n + 1, dtype=np.uint32)
    nc = ctypes.c_uint64(0)
    st = load_library().rc_cohorts_from_batches(_ptr(b) if n else None, n, int(n_batches),
                                                int(max_cohort), _ptr(order), _ptr(offsets),
                                                ctypes.byref(nc))
    if check:
        _check(st, "rc_cohorts_from_batches")
    if st != RC_OK:
        return st
    c = nc.value
    return order[:offsets[c]].copy(), offsets[:c + 1].copy()


# ---------------------------------------------------------------------------
# Device buffers (torch) for one handle
# ---------------------------------------------------------------------------
def _to_device_u32(arr: np.ndarray, device):
    import torch
    return torch.from_numpy(np.ascontiguousarray(arr, dtype=np.uint32).view(np.int32)).to(device)


def _to_host_u32(t) -> np.ndarray:
    return t.cpu().numpy().view(np.uint32)


def buffers_of(tensors: Dict[str, "object"], ld: int, n_words: Optional[int] = None,
               n_steps: Optional[int] = None, n_cohorts: Optional[int] = None) -> RcBuffers:
    """An ``RcBuffers`` pointing at torch tensors (keys as in the C struct).
    Every tensor must be contiguous with 4-byte elements; given the shape
    (W, T, C), each must also hold at least its extent for chains of up to
    T steps (the library checks only that a buffer lies inside one device
    allocation)."""
    need = {"state": None if n_words is None else n_words * ld, "outcome": ld,
            "eff_sid": None if n_steps is None else n_steps * ld,
            "eff_tool": None if n_steps is None else n_steps * ld,
            "eff_payload": None if n_steps is None else 4 * n_steps * ld,
            "n_taken": None if n_steps is None or n_cohorts is None else n_steps * n_cohorts}
    for k, n in need.items():
        t = tensors[k]
        if not t.is_contiguous() or t.element_size() != 4:
            raise ValueError("buffer %s must be a contiguous tensor of 4-byte elements" % k)
        if n is not None and t.numel() < n:
            raise ValueError("buffer %s holds %d elements, needs %d" % (k, t.numel(), n))
    return RcBuffers(tensors["state"].data_ptr(), tensors["outcome"].data_ptr(),
                     tensors["eff_sid"].data_ptr(), tensors["eff_tool"].data_ptr(),
                     tensors["eff_payload"].data_ptr(), tensors["n_taken"].data_ptr(), ld)


class Cohort:
    """A handle plus torch device buffers sized for chains of up to
    ``max_steps`` steps.  State and outcome are uploaded from host arrays
    (uint32, ``[W][ld]`` and ``[ld]``)."""

    def __init__(self, *, n_words, n_routes, cohort_offsets, table, route_mode, route_cdf,
                 decide_thr, max_steps, ld=None, device=0, fill=0xFFFFFFFF):
        import torch
        self.device = torch.device("cuda", device)
        off = _u32(cohort_offsets)
        self.n_sessions = int(off[-1])
        self.n_cohorts = off.size - 1
        self.n_words = n_words
        self.ld = self.n_sessions if ld is None else ld
        self.max_steps = max_steps
        self.handle = rc_cohort_create(n_sessions=self.n_sessions, n_words=n_words,
                                       n_routes=n_routes, cohort_offsets=off, table=table,
                                       route_mode=route_mode, route_cdf=route_cdf,
                                       decide_thr=decide_thr, device=device)
        fill32 = np.uint32(fill).view(np.int32).item()
        T, ld, C = max_steps, self.ld, self.n_cohorts
        mk = lambda *shape: torch.full(shape, fill32, dtype=torch.int32, device=self.device)
        self.t = {"state": mk(n_words, ld), "outcome": mk(ld), "eff_sid": mk(T, ld),
                  "eff_tool": mk(T, ld), "eff_payload": mk(T, ld, 4), "n_taken": mk(T, C)}
        self.buffers = buffers_of(self.t, ld, n_words, T, C)

    @classmethod
    def from_inputs(cls, inp, max_steps=None, device=0):
        c = cls(n_words=inp.n_words, n_routes=inp.n_routes, cohort_offsets=inp.cohort_offsets,
                table=inp.table, route_mode=inp.route_mode, route_cdf=inp.route_cdf,
                decide_thr=inp.decide_thr, max_steps=max_steps or inp.n_steps, ld=inp.ld,
                device=device)
        c.upload(inp.state, inp.outcome)
        return c

    def upload(self, state: np.ndarray, outcome: np.ndarray):
        assert state.shape == (self.n_words, self.ld) and outcome.shape == (self.ld,)
        self.t["state"].copy_(_to_device_u32(state, self.device))
        self.t["outcome"].copy_(_to_device_u32(outcome, self.device))

    def run_chain(self, step0, n_steps, mode=RC_MODE_RESIDENT, cohort_begin=0, cohort_end=None,
                  stream=None):
        assert n_steps <= self.max_steps
        ce = self.n_cohorts if cohort_end is None else cohort_end
        return rc_cohort_run_chain(self.handle, self.buffers, step0, n_steps, mode, cohort_begin,
                                   ce, stream)

    def run_chain_noalloc(self, step0, n_steps, mode=RC_MODE_RESIDENT, cohort_begin=0,
                          cohort_end=None, stream=None):
        assert n_steps <= self.max_steps
        ce = self.n_cohorts if cohort_end is None else cohort_end
        return rc_cohort_run_chain_noalloc(self.handle, self.buffers, step0, n_steps, mode,
                                           cohort_begin, ce, stream)

    def run_floor(self, decisions: np.ndarray, n_steps, cohort_begin=0, cohort_end=None,
                  stream=None):
        """The no-decision floor with a host ``[n_steps][ceil(ld/32)]`` uint32
        decision bitmap (uploaded to the device first)."""
        assert n_steps <= self.max_steps
        bits = np.ascontiguousarray(decisions, dtype=np.uint32)
        assert bits.shape == (n_steps, (self.ld + 31) // 32)
        self.t_bits = _to_device_u32(bits, self.device)
        ce = self.n_cohorts if cohort_end is None else cohort_end
        return rc_cohort_run_floor(self.handle, self.buffers, self.t_bits.data_ptr(), n_steps,
                                   cohort_begin, ce, stream)

    def step(self, step, cohort_begin=0, cohort_end=None, stream=None):
        ce = self.n_cohorts if cohort_end is None else cohort_end
        return rc_cohort_step(self.handle, self.buffers, step, cohort_begin, ce, stream)

    def download(self, n_steps=None) -> Dict[str, np.ndarray]:
        import torch
        torch.cuda.synchronize(self.device)
        T = self.max_steps if n_steps is None else n_steps
        return {"state": _to_host_u32(self.t["state"]), "outcome": _to_host_u32(self.t["outcome"]),
                "eff_sid": _to_host_u32(self.t["eff_sid"][:T]),
                "eff_tool": _to_host_u32(self.t["eff_tool"][:T]),
                "eff_payload": _to_host_u32(self.t["eff_payload"][:T]),
                "n_taken": _to_host_u32(self.t["n_taken"][:T])}

    def last_counts(self):
        return rc_cohort_last_counts(self.handle)

    def plan_info(self):
        return rc_cohort_plan_info(self.handle)

    def close(self):
        if self.handle is not None:
            rc_cohort_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
