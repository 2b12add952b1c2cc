"""Pins of the signed-transform oracle EDT(M) - EDT(not M): closed forms,
the sign and size properties every signed field has, antisymmetry, and
scipy.ndimage.distance_transform_edt as a black box."""
import numpy as np
import pytest

from oracle import edt_oracle


def rand_mask(shape, p_bg, seed):
    rng = np.random.default_rng(seed)
    return (rng.random(shape) >= p_bg).astype(np.uint8)


def test_half_space_closed_form():
    # foreground from row k on: +(x0 - k + 1) there, -(k - x0) above
    shape, k = (9, 5, 4), 3
    m = np.zeros((1,) + shape, np.uint8)
    m[0, k:] = 1
    x0 = np.arange(shape[0]).reshape(-1, 1, 1) * np.ones(shape)
    want = np.where(x0 >= k, x0 - k + 1, -(k - x0)).astype(np.float32)
    assert np.array_equal(edt_oracle.signed_edt(m, 3)[0], want)


def test_single_foreground_element():
    m = np.zeros((1, 7, 6), np.uint8)
    m[0, 2, 4] = 1
    d = np.sqrt(((np.indices((7, 6)) - np.array([2, 4]).reshape(2, 1, 1)) ** 2).sum(0))
    want = -d.astype(np.float32)
    want[2, 4] = 1.0
    assert np.array_equal(edt_oracle.signed_edt(m, 2)[0], want)


def test_sign_size_and_antisymmetry():
    for seed in range(4):
        m = rand_mask((2, 11, 9, 6), 0.3, seed)
        s = edt_oracle.signed_edt(m, 3)
        assert np.all((s > 0) == (m != 0))
        assert np.all(np.abs(s) >= 1.0)
        inv = (m == 0).astype(np.uint8)
        assert np.array_equal(edt_oracle.signed_edt(inv, 3), -s)


def test_one_class_samples_use_the_virtual_element():
    grid = np.indices((4, 5))
    v = np.sqrt((grid[0] + 1.0) ** 2 + grid[1] ** 2).astype(np.float32)
    assert np.array_equal(edt_oracle.signed_edt(np.ones((1, 4, 5), np.uint8), 2)[0], v)
    assert np.array_equal(edt_oracle.signed_edt(np.zeros((1, 4, 5), np.uint8), 2)[0], -v)


def test_scipy_black_box():
    ndi = pytest.importorskip("scipy.ndimage")
    for seed, shape in enumerate([(30,), (13, 17), (6, 7, 9), (3, 4, 5, 6)]):
        m = rand_mask((1,) + shape, 0.25, seed)
        m.flat[0] = 0
        m.flat[-1] = 1
        want = (ndi.distance_transform_edt(m[0]) - ndi.distance_transform_edt(1 - m[0]))
        got = edt_oracle.signed_edt(m, len(shape))[0]
        assert np.allclose(got, want, rtol=1e-6, atol=1e-6), shape
