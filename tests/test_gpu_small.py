"""GPU parity of the one-launch path for small 2-D samples (both extents at
most 64): distances, squared distances and canonical indices must equal the
oracle's exactly, including samples without background (virtual element),
all-background samples, single zeros, one-element and one-row extents, and
batches of mixed samples.  The kernel names show that this path ran; one
size past 64 takes the two-pass path instead."""
import numpy as np
import pytest

from gpu_util import announce, check_against_oracle, run_gpu
from oracle import edt_oracle

pytestmark = pytest.mark.gpu


def run_named(mask, idx=True, sq=True):
    from paper_2608_24738_amd import binding
    binding.prof_enable(64)
    try:
        res = run_gpu(mask, 2, None, dist=True, idx=idx, sq=sq)
        names = [n for n, _ in binding.prof_read()]
    finally:
        binding.prof_enable(0)
    return res, names


def parity_small(mask, tag, idx=True, sq=True, expect="small2d"):
    announce("small 2-D %s shape=%s" % (tag, mask.shape))
    res, names = run_named(mask, idx=idx, sq=sq)
    ora = edt_oracle.edt(mask, 2, None, nthreads=8)
    check_against_oracle(mask, 2, None, res, ora)
    if expect == "small2d":
        assert names and all(n == "small2d" for n in names), names
    else:
        assert "small2d" not in names, names


@pytest.mark.parametrize("shape", [(1, 1), (1, 64), (64, 1), (7, 13), (64, 64), (33, 64), (64, 40), (2, 3)])
@pytest.mark.parametrize("p_bg", [0.02, 0.3])
def test_shapes_and_densities(shape, p_bg):
    rng = np.random.default_rng(shape[0] * 100 + shape[1] + int(p_bg * 100))
    mask = (rng.random((5,) + shape) >= p_bg).astype(np.uint8)
    parity_small(mask, "p_bg=%g" % p_bg)


def test_degenerate_samples():
    mask = np.ones((6, 64, 64), np.uint8)
    mask[0] = 0                     # all background
    # mask[1]: no background (virtual element (-1, 0))
    mask[2, 63, 0] = 0              # one zero in a corner
    mask[3, :, 31] = 0              # one background column
    mask[4, 17] = 0                 # one background row
    mask[5, 0, 0] = mask[5, 63, 63] = 0   # two far zeros: ties along the anti-diagonal
    parity_small(mask, "degenerate")


def test_ties_take_the_smallest_flat_index():
    """Symmetric zeros around every element: equal distances everywhere."""
    mask = np.ones((2, 41, 41), np.uint8)
    mask[0, 10, 10] = mask[0, 10, 30] = mask[0, 30, 10] = mask[0, 30, 30] = 0
    mask[1, ::4, ::4] = 0
    parity_small(mask, "ties")


def test_outputs_one_at_a_time():
    rng = np.random.default_rng(9)
    mask = (rng.random((3, 50, 60)) >= 0.05).astype(np.uint8)
    parity_small(mask, "dist only", idx=False, sq=False)
    parity_small(mask, "dist + idx", idx=True, sq=False)


def test_large_batch():
    rng = np.random.default_rng(10)
    mask = (rng.random((300, 64, 64)) >= 0.1).astype(np.uint8)
    mask[::7] = 1                   # some samples without background
    parity_small(mask, "batch 300")


def test_past_64_takes_the_two_pass_path():
    rng = np.random.default_rng(11)
    mask = (rng.random((2, 65, 64)) >= 0.05).astype(np.uint8)
    parity_small(mask, "65 rows", expect="other")
