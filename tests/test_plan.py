"""The launch plan (host logic, CPU only): every session is processed by
exactly one lane, in a lane that knows its cohort, with the packing rules
the compaction relies on."""
import numpy as np
import pytest

from paper_2608_12123_amd import rc_cohort as rc
from paper_2608_12123_amd import workload as wk

NONE = 0xFFFFFFFF


def check_plan(sizes, lanes_per_wg):
    sizes = np.asarray(sizes, dtype=np.int64)
    off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.uint32)
    N = int(off[-1])
    ses, coh = rc.rc_plan_lanes(cohort_offsets=off, lanes_per_workgroup=lanes_per_wg)
    assert ses.size % lanes_per_wg == 0
    act = ses != NONE
    # every session exactly once
    counts = np.bincount(ses[act].astype(np.int64), minlength=N)
    assert counts.size == N and np.all(counts == 1)
    # each lane's cohort contains its session
    c = coh[act].astype(np.int64)
    s = ses[act].astype(np.int64)
    assert np.all(off[c] <= s) and np.all(s < off[c + 1])
    waves = ses.reshape(-1, 64)
    cw = coh.reshape(-1, 64)
    for w in range(waves.shape[0]):
        a = waves[w] != NONE
        if not a.any():
            continue
        n_act = int(a.sum())
        # active lanes are a prefix
        assert a[:n_act].all() and not a[n_act:].any()
        for cc in np.unique(cw[w][:n_act]):
            k = int(off[cc + 1] - off[cc])
            lanes = np.flatnonzero(cw[w][:n_act] == cc)
            # each cohort's lanes are one run holding its sessions in order
            assert np.all(np.diff(lanes) == 1)
            assert np.all(np.diff(waves[w][lanes].astype(np.int64)) == 1)
            # small cohorts lie wholly inside this wavefront
            if k <= 64:
                assert lanes.size == k
    # a large cohort starts at lane 0 of a wavefront, spans consecutive
    # wavefronts of one workgroup
    lane_idx = {int(x): i for i, x in enumerate(ses) if x != NONE}
    for cc in np.nonzero(sizes > 64)[0]:
        first = lane_idx[int(off[cc])]
        last = lane_idx[int(off[cc + 1]) - 1]
        assert first % 64 == 0
        assert first // lanes_per_wg == last // lanes_per_wg
        assert last - first + 1 == sizes[cc]
    return ses.size


def rand_sizes(seed, n, kinds):
    rng = np.random.Generator(np.random.PCG64(seed))
    return rng.choice(kinds, size=n)


@pytest.mark.parametrize("lanes", [256, 512])
@pytest.mark.parametrize("seed", range(6))
def test_random_mixes(seed, lanes):
    kinds = [[1, 2, 3, 5, 17, 31, 32, 33, 63, 64, 65, 100, 127, 128, 129, 200, 255, 256],
             [32, 64, 128, 256], [1, 7, 64, 256], [256], [32], [65, 129, 193]][seed]
    check_plan(rand_sizes(seed, 700, kinds), lanes)


@pytest.mark.parametrize("lanes", [256, 512])
def test_variable_1m_workload(lanes):
    inp = wk.make_inputs(wk.WORKLOADS["s1m"])
    n_lanes = check_plan(np.diff(inp.cohort_offsets.astype(np.int64)), lanes)
    assert n_lanes < 1.05 * inp.n_sessions  # first fit wastes little


def test_bins_of_cohort_ranges():
    """Small cohorts go, in order, to the open bin or a later one; a large
    cohort lands at most one bin before the bin of any earlier large cohort
    (the two most recent bins stay open).  So a cohort range maps to a
    contiguous range of bins, widened by one on each side for large ones."""
    rng = np.random.Generator(np.random.PCG64(5))
    sizes = rng.choice([1, 5, 17, 31, 32, 64, 65, 128, 192, 256], size=3000)
    off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.uint32)
    for lanes in (256, 512):
        ses, coh = rc.rc_plan_lanes(cohort_offsets=off, lanes_per_workgroup=lanes)
        bin_of = np.full(sizes.size, -1, dtype=np.int64)
        idx = np.flatnonzero(coh != NONE)
        bin_of[coh[idx].astype(np.int64)] = idx // lanes
        assert (bin_of >= 0).all()
        small = sizes <= 64
        bs = bin_of[small]
        assert np.all(np.diff(bs) >= 0)
        bl = bin_of[~small]
        assert np.all(bl >= np.maximum.accumulate(bl) - 1)
        assert bl.min() > bs.max()  # the classes never share a bin


def test_uniform_workloads():
    check_plan([256] * 390 + [160], 256)
    check_plan([32] * 1000, 256)
    check_plan([64] * 1000, 256)


def test_rejects_bad_arguments():
    off = np.asarray([0, 10], dtype=np.uint32)
    with pytest.raises(rc.RcError):
        rc.rc_plan_lanes(cohort_offsets=off, lanes_per_workgroup=100)
    with pytest.raises(rc.RcError):
        rc.rc_plan_lanes(cohort_offsets=np.asarray([0, 300], dtype=np.uint32))
