"""The C-ABI library: it loads, exports every symbol the header declares,
and rejects bad arguments before touching a device (CPU only)."""
import ctypes
import os
import re

import numpy as np
import pytest

from paper_2608_12123_amd import rc_cohort as rc

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "rc_cohort.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:int|const char\s*\*)\s*(rc_\w+)\s*\(", text, flags=re.M)))


@pytest.fixture(scope="module")
def lib():
    return rc.load_library()


def test_header_declares_the_boundary():
    names = declared_functions()
    for must in ("rc_cohort_create", "rc_cohort_step", "rc_cohort_run_chain", "rc_cohort_destroy"):
        assert must in names
    assert sorted(rc.EXPORTED) == names


def test_binding_limits_match_the_header():
    text = open(HEADER).read()
    defs = dict(re.findall(r"^#define\s+(RC_(?:MIN|MAX)_\w+)\s+\(?(\w+)", text, flags=re.M))
    assert sorted(defs) == ["RC_MAX_COHORT", "RC_MAX_ROUTES", "RC_MAX_SESSIONS", "RC_MAX_WORDS",
                            "RC_MIN_WORDS"]
    shift = re.search(r"^#define\s+RC_MAX_SESSIONS\s+\(1u\s*<<\s*(\d+)\)", text, flags=re.M)
    values = {k: int(v.rstrip("u")) for k, v in defs.items() if k != "RC_MAX_SESSIONS"}
    values["RC_MAX_SESSIONS"] = 1 << int(shift.group(1))
    for k, v in values.items():
        assert getattr(rc, k) == v, k


def test_library_exports_every_declared_symbol(lib):
    for name in declared_functions():
        assert hasattr(lib, name), name
        assert hasattr(rc, name), "binding lacks " + name


def test_status_strings(lib):
    assert [rc.rc_status_string(i) for i in range(4)] == [
        "RC_OK", "RC_E_INVALID", "RC_E_NOMEM", "RC_E_DEVICE"]
    assert rc.rc_status_string(99) == "RC_E_UNKNOWN"


def test_null_handles(lib):
    assert lib.rc_cohort_destroy(None) == rc.RC_OK
    assert lib.rc_cohort_run_chain(None, None, 0, 1, 0, 0, 1, None) == rc.RC_E_INVALID
    assert lib.rc_cohort_step(None, None, 0, 0, 1, None) == rc.RC_E_INVALID
    assert lib.rc_cohort_run_chain_noalloc(None, None, 0, 1, 1, 0, 1, None) == rc.RC_E_INVALID
    assert lib.rc_cohort_last_counts(None, None, None) == rc.RC_E_INVALID
    assert lib.rc_cohort_plan_info(None, None, None, None) == rc.RC_E_INVALID


def good_desc():
    return dict(n_sessions=100, n_words=8, n_routes=4,
                cohort_offsets=np.asarray([0, 32, 64, 100], dtype=np.uint32),
                table=np.arange(64, dtype=np.uint32), route_mode=rc.RC_ROUTE_MOD,
                route_cdf=None, decide_thr=32768)


BAD = {
    "no_sessions": dict(n_sessions=0, cohort_offsets=[0]),
    "too_few_words": dict(n_words=3),
    "too_many_words": dict(n_words=65),
    "no_routes": dict(n_routes=0),
    "too_many_routes": dict(n_routes=1025, table=np.zeros(1025 * 16, dtype=np.uint32)),
    "offsets_not_from_zero": dict(cohort_offsets=[1, 32, 64, 100]),
    "offsets_not_to_n": dict(cohort_offsets=[0, 32, 64, 99]),
    "empty_cohort": dict(cohort_offsets=[0, 32, 32, 100]),
    "decreasing_offsets": dict(cohort_offsets=[0, 64, 32, 100]),
    "cohort_too_big": dict(n_sessions=300, cohort_offsets=[0, 257, 300]),
    "threshold_too_big": dict(decide_thr=65537),
    "bad_route_mode": dict(route_mode=2),
    "cdf_missing": dict(route_mode=rc.RC_ROUTE_CDF, route_cdf=None),
    "cdf_decreasing": dict(route_mode=rc.RC_ROUTE_CDF, route_cdf=[5, 4, 9]),
}


@pytest.mark.parametrize("name", sorted(BAD))
def test_invalid_descriptor_rejected_before_device(lib, name):
    d = good_desc()
    d.update(BAD[name])
    st, h = rc.rc_cohort_create(**d, check=False)
    assert st == rc.RC_E_INVALID, rc.rc_status_string(st)
    assert not h.value


def test_null_out_pointer(lib):
    d = good_desc()
    off = np.asarray(d["cohort_offsets"], dtype=np.uint32)
    tab = np.asarray(d["table"], dtype=np.uint32)
    desc = rc.RcCohortDesc(100, 8, 4, 3, off.ctypes.data_as(rc._P32), tab.ctypes.data_as(rc._P32),
                           0, None, 32768)
    assert lib.rc_cohort_create(ctypes.byref(desc), 0, None) == rc.RC_E_INVALID
    assert lib.rc_cohort_create(None, 0, ctypes.byref(ctypes.c_void_p())) == rc.RC_E_INVALID


def _has_gpu():
    try:
        import torch
        return torch.cuda.is_available()
    except Exception:
        return False


@pytest.mark.skipif(_has_gpu(), reason="checks the no-device path")
def test_valid_descriptor_without_device_is_device_error(lib):
    st, h = rc.rc_cohort_create(**good_desc(), check=False)
    assert st == rc.RC_E_DEVICE
    assert not h.value


def plan_lanes_status(lib, d):
    """rc_plan_lanes on a full descriptor (host only: the same descriptor
    checks as rc_cohort_create, no device involved)."""
    off = np.ascontiguousarray(d["cohort_offsets"], dtype=np.uint32)
    tab = np.ascontiguousarray(d["table"], dtype=np.uint32)
    cdf = None if d["route_cdf"] is None else np.ascontiguousarray(d["route_cdf"], dtype=np.uint32)
    desc = rc.RcCohortDesc(d["n_sessions"], d["n_words"], d["n_routes"], off.size - 1,
                           off.ctypes.data_as(rc._P32), tab.ctypes.data_as(rc._P32),
                           d["route_mode"], None if cdf is None else cdf.ctypes.data_as(rc._P32),
                           d["decide_thr"])
    n = ctypes.c_uint32()
    return lib.rc_plan_lanes(ctypes.byref(desc), 256, None, None, 0, ctypes.byref(n))


@pytest.mark.parametrize("name", sorted(BAD))
def test_invalid_descriptor_rejected_by_plan_inspection(lib, name):
    d = good_desc()
    d.update(BAD[name])
    assert plan_lanes_status(lib, d) == rc.RC_E_INVALID
    assert plan_lanes_status(lib, good_desc()) == rc.RC_OK
