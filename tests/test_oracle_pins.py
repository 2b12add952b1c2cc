"""The CPU oracle against what the paper and mathematics fix (no GPU)."""
import numpy as np
import pytest

import pins
from oracle import edt_oracle


@pytest.fixture(scope="module")
def orc():
    return edt_oracle.default()


@pytest.mark.parametrize("pin", pins.ALL_PINS, ids=lambda f: f.__name__)
def test_pin(orc, pin):
    pin(orc)


def test_threads_do_not_change_results(orc):
    rng = np.random.default_rng(3)
    mask = (rng.random((3, 9, 10, 11)) >= 0.2).astype(np.uint8)
    a = orc.edt(mask, ndim=3, nthreads=1)
    b = orc.edt(mask, ndim=3, nthreads=4)
    for k in ("sq", "dist", "idx"):
        assert np.array_equal(a[k], b[k])


def test_rejects_bad_arguments(orc):
    m = np.ones((1, 4, 4), np.uint8)
    with pytest.raises(ValueError):
        orc.edt(m, sampling=(1.0, 0.0))
    with pytest.raises(ValueError):
        orc.edt(m, sampling=(1.0, float("nan")))
    with pytest.raises(ValueError):
        orc.edt(np.ones((1,) + (1,) * 9, np.uint8))


def test_scipy_cross_check(orc):
    """Optional black-box agreement with scipy.ndimage where it is installed:
    squared distances after rounding, indices by validity only (scipy's tie
    choice is not canonical)."""
    ndi = pytest.importorskip("scipy.ndimage")
    from invariants import check_index_valid
    rng = np.random.default_rng(17)
    for trial in range(20):
        nd = 1 + trial % 3
        shape = tuple(int(rng.integers(1, 12)) for _ in range(nd))
        mask = (rng.random(shape) >= 0.25).astype(np.uint8)
        if not (mask == 0).any():
            continue
        d, i = ndi.distance_transform_edt(mask, return_indices=True)
        r = orc.edt(mask[None])
        assert np.array_equal(np.rint(d * d).astype(np.int64), r["sq"][0])
        assert check_index_valid(mask, r["sq"][0], i) == 0
        samp = tuple(float(x) for x in rng.uniform(0.5, 2.0, nd))
        d = ndi.distance_transform_edt(mask, sampling=samp)
        r = orc.edt(mask[None], sampling=samp)
        assert np.allclose(r["sqd"][0], d * d, rtol=1e-12, atol=1e-12)
