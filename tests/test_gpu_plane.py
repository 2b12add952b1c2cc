"""GPU parity of the plane-ordered path (unit sampling, distance outputs,
rank 3 with the last two extents both 128, or both 64 with an even number of
planes per sample): axis-0 nearest-zero scan from the mask, then one
workgroup per 128 x 128 plane or pair of 64 x 64 planes.  Squared distances and
distances must equal the oracle's bit for bit; the kernel names the library
reports show which path ran."""
import numpy as np
import pytest

from gpu_util import announce, check_against_oracle, run_gpu
from oracle import edt_oracle
from paper_2608_24738_amd import workloads

pytestmark = pytest.mark.gpu


def rand_mask(shape, p_bg, seed):
    rng = np.random.default_rng(seed)
    return (rng.random(shape) >= p_bg).astype(np.uint8)


def run_and_names(mask, ndim, dist=True, sq=True):
    from paper_2608_24738_amd import binding
    binding.prof_enable(64)
    try:
        res = run_gpu(mask, ndim, None, dist=dist, idx=False, sq=sq)
        names = [n for n, _ in binding.prof_read()]
    finally:
        binding.prof_enable(0)
    return res, names


def parity_plane(mask, ndim, tag, dist=True, sq=True, expect_plane=True):
    announce("plane %s shape=%s dist=%s sq=%s" % (tag, mask.shape, dist, sq))
    res, names = run_and_names(mask, ndim, dist=dist, sq=sq)
    ora = edt_oracle.edt(mask, ndim, None, nthreads=16)
    check_against_oracle(mask, ndim, None, res, ora)
    if expect_plane:
        # 3-D: the axis-0 distances reach the plane pass as bytes; with middle
        # axes they travel as 16-bit squares
        fmt = ("o8", "i8") if mask.shape[-1] == 128 else ("o16", "i16")
        assert "col_scan." + fmt[0] in names and "plane_final." + fmt[1] in names, names
        assert not any(n.startswith(("plane_pair", "scan_")) for n in names), names
    else:
        assert not any(n.startswith("plane_final") for n in names), names
    return names


# axis-0 extents from 1 to 128 (8 waves of 16 rows, ragged last chunk)
@pytest.mark.parametrize("n0", [1, 2, 7, 16, 17, 64, 100, 128])
def test_axis0_extents(n0):
    mask = rand_mask((2, n0, 128, 128), 0.02, 100 + n0)
    parity_plane(mask, 3, "n0=%d" % n0)


@pytest.mark.parametrize("p_bg", [0.0005, 0.05, 0.5, 0.95])
def test_densities(p_bg):
    mask = rand_mask((3, 32, 128, 128), p_bg, int(p_bg * 1e4))
    parity_plane(mask, 3, "p_bg=%g" % p_bg)


def test_balls_twin():
    """The headline structure (foreground = union of balls) at 48 x 128^2."""
    mask = workloads.make_mask(3, (48, 128, 128), 3)
    parity_plane(mask, 3, "balls")


def test_squared_only_and_distance_only():
    mask = rand_mask((2, 40, 128, 128), 0.01, 5)
    parity_plane(mask, 3, "sq only", dist=False, sq=True)
    parity_plane(mask, 3, "dist only", dist=True, sq=False)


def test_degenerate_samples():
    """All background, no background (virtual element), a single zero, a
    single zero column, and whole planes without background."""
    shape = (6, 20, 128, 128)
    mask = np.ones(shape, np.uint8)
    mask[0] = 0                               # all background
    # mask[1]: no background at all (virtual element (-1, 0, ..., 0))
    mask[2, 19, 127, 0] = 0                   # one zero in a corner
    mask[3, :, 64, 65] = 0                    # one column of zeros along axis 0
    mask[4, 0, 5, 7] = 0                      # a zero in the first plane only
    mask[5, 10] = 0                           # one whole background plane
    parity_plane(mask, 3, "degenerate")


def test_four_dims_keep_the_other_path():
    """Rank 4 with 128 x 128 planes runs the last-axis-first order."""
    parity_plane(rand_mask((2, 9, 5, 128, 128), 0.003, 44), 4, "4-D", expect_plane=False)
    parity_plane(workloads.make_mask(5, (6, 3, 128, 128), 2), 4, "4-D sparse", expect_plane=False)


def test_fallbacks_keep_the_other_path():
    """Inputs outside the plane path's limits take the other kernels."""
    parity_plane(rand_mask((1, 129, 128, 128), 0.01, 3), 3, "n0=129", expect_plane=False)
    parity_plane(rand_mask((1, 8, 64, 128), 0.01, 4), 3, "64x128 planes", expect_plane=False)


def test_full_headline_with_squares():
    """8 x 128^3 balls: exact squared distances and distances in one call."""
    mask = workloads.make_mask(3)
    parity_plane(mask, 3, "headline")


# ---- 64 x 64 planes (two per workgroup, 16-bit runs of half-run rows) -------
@pytest.mark.parametrize("n0", [2, 6, 64, 128])
def test_planes_64(n0):
    mask = rand_mask((3, n0, 64, 64), 0.01, 200 + n0)
    parity_plane(mask, 3, "64 n0=%d" % n0)


def test_planes_64_structures():
    parity_plane(workloads.make_mask(11), 3, "8x64^3 balls")
    parity_plane(workloads.make_mask(5, (24, 64, 64), 2), 3, "sparse background")


def test_planes_64_degenerate_and_odd():
    shape = (4, 8, 64, 64)
    mask = np.ones(shape, np.uint8)
    mask[0] = 0                               # all background
    # mask[1]: no background (virtual element)
    mask[2, 7, 63, 0] = 0
    mask[3, :, 31, 32] = 0
    parity_plane(mask, 3, "64 degenerate")
    # an odd number of planes per sample keeps the other path
    parity_plane(rand_mask((2, 5, 64, 64), 0.02, 9), 3, "64 odd planes", expect_plane=False)



# Workgroup b takes plane b * m mod planes: plane counts divisible by the
# first multiplier the host tries (397), and ones that are not, including
# counts below it.  Every plane must be written exactly once with its own
# result, including samples without background (virtual element).
@pytest.mark.parametrize("batch,n0", [(397, 1), (3, 97), (1, 1), (5, 79)])
def test_plane_permutation_counts(batch, n0):
    mask = rand_mask((batch, n0, 128, 128), 0.01, 4000 + batch + n0)
    mask[0] = 1
    parity_plane(mask, 3, "planes=%d" % (batch * n0))
