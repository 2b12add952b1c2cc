"""Pins of the chamfer-transform oracle and of the point-wise spot check.

The chamfer oracle is the brute-force taxicab / chessboard value (pinned in
test_oracle_bf.py) with -1 for samples without background.  Here it is held
against closed forms and against scipy.ndimage.distance_transform_cdt, an
independent chamfer-sweep implementation, as a black box."""
import numpy as np
import pytest

from invariants import chamfer_fixed_point_violations
from oracle import edt_oracle
from paper_2608_24738_amd import workloads

CHAMFER = ("taxicab", "chessboard")


def rand_mask(shape, p_bg, seed):
    rng = np.random.default_rng(seed)
    return (rng.random(shape) >= p_bg).astype(np.uint8)


@pytest.mark.parametrize("metric", CHAMFER)
def test_single_zero_closed_form(metric):
    shape, c = (6, 5, 7), (2, 4, 3)
    m = np.ones((1,) + shape, np.uint8)
    m[(0,) + c] = 0
    d = np.abs(np.indices(shape) - np.array(c).reshape(3, 1, 1, 1))
    want = d.sum(0) if metric == "taxicab" else d.max(0)
    got = edt_oracle.cdt(m, 3, metric)
    assert got.dtype == np.int32
    assert np.array_equal(got[0], want)


@pytest.mark.parametrize("metric", CHAMFER)
def test_no_background_is_minus_one(metric):
    m = np.ones((3, 4, 5), np.uint8)
    m[1, 2, 2] = 0                                   # only the middle sample has background
    got = edt_oracle.cdt(m, 2, metric)
    assert np.all(got[0] == -1) and np.all(got[2] == -1)
    assert got[1, 2, 2] == 0 and got[1].min() == 0
    assert np.all(edt_oracle.cdt(np.zeros((1, 3, 3), np.uint8), 2, metric) == 0)


@pytest.mark.parametrize("metric", CHAMFER)
def test_scipy_black_box(metric):
    ndi = pytest.importorskip("scipy.ndimage")
    cases = [((23,), 0.1), ((1,), 0.0), ((9, 14), 0.05), ((1, 17), 0.2), ((6, 7, 5), 0.03),
             ((4, 3, 5, 6), 0.02), ((5, 4), 0.0), ((3, 2, 2, 2, 3), 0.1)]
    for seed, (shape, p) in enumerate(cases):
        m = rand_mask((2,) + shape, p, seed)
        got = edt_oracle.cdt(m, len(shape), metric)
        for b in range(2):
            want = ndi.distance_transform_cdt(m[b], metric=metric)
            assert np.array_equal(got[b], want), (metric, shape, b)


@pytest.mark.parametrize("metric", ("euclidean",) + CHAMFER)
def test_point_spot_check_matches_whole_transform(metric):
    m = rand_mask((1, 13, 11, 6), 0.04, 7)
    m[0, 12, 10, 5] = 0
    whole = edt_oracle.dt_bf(m, 3, metric, want_idx=False)["value"][0]
    rng = np.random.default_rng(3)
    pts = np.stack([rng.integers(0, n, 40) for n in (13, 11, 6)], axis=1)
    got = edt_oracle.metric_dt_at(m[0], metric, pts)
    assert np.array_equal(got, whole[tuple(pts.T)])
    assert np.all(np.isnan(edt_oracle.metric_dt_at(np.ones((4, 4), np.uint8), metric, [[1, 2]])))


def test_point_spot_check_closed_form():
    s = np.ones((9, 9), np.uint8)
    s[4, 4] = 0
    pts = np.array([[0, 0], [4, 4], [8, 3], [1, 7]])
    d = np.abs(pts - 4)
    assert np.array_equal(edt_oracle.metric_dt_at(s, "euclidean", pts), (d * d).sum(1))
    assert np.array_equal(edt_oracle.metric_dt_at(s, "taxicab", pts), d.sum(1))
    assert np.array_equal(edt_oracle.metric_dt_at(s, "chessboard", pts), d.max(1))


@pytest.mark.parametrize("metric", CHAMFER)
def test_fixed_point_check_accepts_the_oracle_and_nothing_near_it(metric):
    # the full-size GPU check: it must pass the oracle and fail a field one
    # off anywhere, the other metric's field and a field without -1
    m = workloads.make_mask(8, (48, 56), 2)
    d = edt_oracle.cdt(m, 2, metric)
    other = "chessboard" if metric == "taxicab" else "taxicab"
    for b in range(2):
        assert chamfer_fixed_point_violations(m[b, 0], d[b, 0], metric) == 0
        assert chamfer_fixed_point_violations(m[b, 0], d[b, 0], other) > 0
    rng = np.random.default_rng(1)
    for _ in range(20):
        e = d[0, 0].copy()
        k = tuple(int(rng.integers(0, n)) for n in e.shape)
        e[k] += int(rng.choice([-1, 1]))
        assert chamfer_fixed_point_violations(m[0, 0], e, metric) > 0, k
    assert chamfer_fixed_point_violations(np.ones((4, 5), np.uint8), np.full((4, 5), -1), metric) == 0
    assert chamfer_fixed_point_violations(np.ones((4, 5), np.uint8), np.zeros((4, 5)), metric) > 0
