"""GPU parity of the tiled passes on the index carrier (k_tile_idx) in each of
their forms: rank 2 and 3 with the rank built in (sampled rank 3 in either
pass order), with shift-and-mask coordinates and 32-bit buffer offsets when
every extent after axis 0 is a power of two and the line length a multiple of
32, or with divisions otherwise; and the generic form for other ranks.  Every
case checks that the
tiled passes ran, and compares with the oracle element by element: unit
sampling bit-exact with the canonical indices, sampled within 1e-5 / 1e-6
with every index a nearest background element.
"""
import numpy as np
import pytest

from gpu_util import announce, check_against_oracle, run_gpu
from oracle import edt_oracle

pytestmark = pytest.mark.gpu

ANISO3 = (2.5, 0.8, 0.8)      # rank 3, axis 0 weighs most: axis 0 runs first, axis 1 last
ANISO3B = (0.8, 2.5, 1.0)     # axis 1 weighs most: the default order (axis 1, then axis 0)


def rand_mask(shape, p_bg, seed):
    rng = np.random.default_rng(seed)
    return (rng.random(shape) >= p_bg).astype(np.uint8)


def parity_tidx(mask, ndim, sampling, dist=True, idx=True, sq=None, tag=""):
    from paper_2608_24738_amd import binding
    unit = sampling is None
    sq = unit if sq is None else sq
    announce("%s shape=%s sampling=%s dist=%s idx=%s sq=%s" % (tag, mask.shape, sampling, dist, idx, sq))
    binding.prof_enable(64)
    try:
        res = run_gpu(mask, ndim, sampling, dist=dist, idx=idx, sq=sq)
        names = {n for n, _ in binding.prof_read()}
    finally:
        binding.prof_enable(0)
    assert "tile_idx_final" in names, "the tiled index pass did not run: %s" % sorted(names)
    ora = edt_oracle.edt(mask, ndim, sampling, nthreads=16)
    check_against_oracle(mask, ndim, sampling, res, ora)


# shift-and-mask coordinates, buffer offsets, 2 x 32 patches
FAST = [
    ((2, 64, 32, 64), 0.01, 3),
    ((1, 32, 64, 128), 0.002, 3),
    ((3, 96, 128), 0.01, 2),
    ((2, 256, 64), 0.001, 2),
]


@pytest.mark.parametrize("shape,p_bg,ndim", FAST, ids=["x".join(map(str, s)) for s, _, _ in FAST])
def test_fast_tiles(shape, p_bg, ndim):
    mask = rand_mask(shape, p_bg, sum(shape))
    samp = ANISO3 if ndim == 3 else (1.7, 0.6)
    parity_tidx(mask, ndim, None, tag="unit")
    parity_tidx(mask, ndim, None, dist=False, idx=True, sq=False, tag="unit, indices only")
    parity_tidx(mask, ndim, samp, tag="sampled")
    # distances only: the flat-index carrier runs inside the distance output
    parity_tidx(mask, ndim, samp, dist=True, idx=False, sq=False, tag="sampled, distances only")
    if ndim == 3:
        parity_tidx(mask, ndim, ANISO3B, tag="sampled, default order")


# divisions for the coordinates (extents that are not powers of two, or line
# lengths that are not multiples of 32), and the generic kernel (rank 4)
GENERAL = [
    ((2, 40, 48, 50), 0.01, 3),
    ((2, 48, 24, 64), 0.01, 3),      # axis-1 lines of 24 rows: not a multiple of 32
    ((3, 70, 90), 0.02, 2),
    ((2, 12, 16, 16, 16), 0.01, 4),
]


@pytest.mark.parametrize("shape,p_bg,ndim", GENERAL, ids=["x".join(map(str, s)) for s, _, _ in GENERAL])
def test_general_tiles(shape, p_bg, ndim):
    mask = rand_mask(shape, p_bg, sum(shape) + 1)
    samp = {2: (1.7, 0.6), 3: ANISO3, 4: (1.3, 2.5, 0.8, 0.8)}[ndim]
    parity_tidx(mask, ndim, None, tag="unit")
    parity_tidx(mask, ndim, samp, tag="sampled")
    parity_tidx(mask, ndim, samp, dist=True, idx=False, sq=False, tag="sampled, distances only")
    if ndim == 3:
        parity_tidx(mask, ndim, ANISO3B, tag="sampled, default order")


def test_longest_searches_and_empty_samples():
    """One background voxel at a far corner (searches run the whole line, up
    to the end of the weight table), next to a sample without background (the
    virtual element) and one of all background."""
    mask = np.ones((3, 64, 64, 64), np.uint8)
    mask[0, 63, 63, 63] = 0
    mask[2] = 0
    parity_tidx(mask, 3, None, tag="corner / none / all")
    parity_tidx(mask, 3, ANISO3, tag="corner / none / all, sampled")
    parity_tidx(mask, 3, ANISO3B, tag="corner / none / all, sampled, default order")
    m2 = np.ones((2, 33, 40, 50), np.uint8)            # the same with divisions
    m2[0, 0, 39, 0] = 0
    parity_tidx(m2, 3, ANISO3, tag="corner / none, divisions, sampled")
    parity_tidx(m2, 3, ANISO3B, tag="corner / none, divisions, sampled, default order")
