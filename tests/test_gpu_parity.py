"""GPU parity: the HIP library against the CPU oracle, element by element.

Unit sampling: int32 squared distances and float distances bit-exact, indices
equal to the canonical ones.  Sampled: distances within 1e-5 relative or
1e-6 absolute, indices checked to be nearest background elements.
"""
import numpy as np
import pytest

from gpu_util import announce, check_against_oracle, run_gpu
from oracle import edt_oracle
from paper_2608_24738_amd import workloads

pytestmark = pytest.mark.gpu

NTHREADS = 16


def oracle(mask, ndim, sampling=None):
    return edt_oracle.edt(mask, ndim, sampling, nthreads=NTHREADS)


def parity(mask, ndim, sampling=None, dist=True, idx=False, sq=None, tag=""):
    unit = sampling is None
    if sq is None:
        sq = unit
    announce("%s shape=%s ndim=%d sampling=%s dist=%s idx=%s sq=%s"
             % (tag, mask.shape, ndim, sampling, dist, idx, sq))
    res = run_gpu(mask, ndim, sampling, dist=dist, idx=idx, sq=sq)
    ora = oracle(mask, ndim, sampling)
    check_against_oracle(mask, ndim, sampling, res, ora)
    return res, ora


# ---- the five workloads at smaller sizes (several tiles, ragged tails) -------
TWINS = [
    (1, (64, 64), 1, True),
    (2, (100, 72), 3, False),        # last axis 72 does not divide the 1024-byte span
    (2, (128, 256), 2, False),
    (3, (40, 37, 64), 3, False),
    (3, (33, 48, 96), 2, True),
    (4, (30, 33, 64), 2, True),
    (4, (17, 40, 52), 1, False),
    (5, (5, 9, 10, 64), 2, False),
    (5, (3, 7, 11, 13), 3, True),
]


@pytest.mark.parametrize("key,spatial,batch,want_idx", TWINS,
                         ids=["cfg%d-%s-b%d%s" % (k, "x".join(map(str, s)), b, "-idx" if i else "")
                              for k, s, b, i in TWINS])
def test_workload_twins(key, spatial, batch, want_idx):
    w = workloads.WORKLOADS[key]
    mask = workloads.make_mask(key, spatial, batch)
    samp = w.sampling
    parity(mask, len(spatial), samp, dist=True, idx=want_idx, tag="twin cfg%d" % key)
    if want_idx:
        # indices alone (no distance output) take the same path
        parity(mask, len(spatial), samp, dist=False, idx=True, sq=False, tag="idx-only cfg%d" % key)


# ---- the five workloads at full size, in the configuration the bench times ---
FULL = [(1, True), (2, False), (3, False), (4, True), (5, False)]


@pytest.mark.parametrize("key,want_idx", FULL, ids=["cfg%d" % k for k, _ in FULL])
def test_workload_full_size(key, want_idx):
    w = workloads.WORKLOADS[key]
    mask = workloads.make_mask(key)
    parity(mask, w.ndim, w.sampling, dist=True, idx=want_idx, tag="full cfg%d" % key)


# ---- edge cases -------------------------------------------------------------
def rand_mask(shape, p_bg, seed):
    rng = np.random.default_rng(seed)
    return (rng.random(shape) >= p_bg).astype(np.uint8)


@pytest.mark.parametrize("ndim", [1, 2, 3, 4, 5, 6, 7, 8])
def test_every_rank(ndim):
    rng = np.random.default_rng(100 + ndim)
    spatial = tuple(int(rng.integers(1, 6 if ndim > 4 else 12)) for _ in range(ndim))
    mask = rand_mask((3,) + spatial, 0.15, ndim)
    parity(mask, ndim, None, dist=True, idx=True, tag="rank")
    parity(mask, ndim, [1.5] * ndim, dist=True, idx=True, tag="rank sampled")
    parity(mask, ndim, [0.5 + 0.25 * a for a in range(ndim)], dist=True, idx=False, tag="rank sampled")


@pytest.mark.parametrize("case", ["all_background", "all_foreground", "single_zero", "unit_extent"])
def test_degenerate_inputs(case):
    shape = (2, 9, 17, 33)
    if case == "all_background":
        mask = np.zeros(shape, np.uint8)
    elif case == "all_foreground":
        mask = np.ones(shape, np.uint8)
    elif case == "single_zero":
        mask = np.ones(shape, np.uint8)
        mask[0, 4, 3, 30] = 0
        mask[1, 8, 16, 0] = 0
    else:
        shape = (4, 1, 7, 1)
        mask = rand_mask(shape, 0.3, 9)
    parity(mask, 3, None, dist=True, idx=True, tag=case)
    parity(mask, 3, (2.5, 0.8, 0.8), dist=True, idx=True, tag=case + " sampled")
    parity(mask, 3, (2.5, 0.8, 0.8), dist=True, idx=False, tag=case + " sampled")


def test_mixed_batch_with_and_without_background():
    mask = rand_mask((5, 21, 30), 0.02, 3)
    mask[1] = 1
    mask[3] = 1
    parity(mask, 2, None, dist=True, idx=True, tag="mixed batch")
    parity(mask, 2, (0.7, 1.3), dist=True, idx=True, tag="mixed batch sampled")


@pytest.mark.parametrize("n", [1, 2, 3, 63, 65, 1000, 1024, 1025, 3000])
def test_scan_line_lengths(n):
    """Rank-1 lines and 2-D last axes of every scan variant (span, generic, long)."""
    mask = rand_mask((3, n), 0.05, n)
    parity(mask, 1, None, dist=True, idx=True, tag="1-D n=%d" % n)
    parity(mask, 1, (1.7,), dist=True, idx=True, tag="1-D sampled n=%d" % n)
    m2 = rand_mask((2, 3, n), 0.02, n + 1)
    parity(m2, 2, None, dist=True, idx=True, tag="2-D n=%d" % n)
    parity(m2, 2, None, dist=True, idx=False, tag="2-D n=%d" % n)


@pytest.mark.parametrize("n", [700, 1500, 3000, 6000])
def test_long_strided_lines(n):
    """Strided lines long enough that fewer than 64 lanes share a workgroup's LDS,
    products that need the int64 comparison path (n >= 3000, sampled), and
    (n = 6000) a whole-line search with 4 lines per workgroup."""
    mask = rand_mask((n, 40), 0.003, n)
    parity(mask[None], 2, None, dist=True, idx=True, tag="long strided n=%d" % n)
    parity(mask[None], 2, None, dist=True, idx=False, tag="long strided n=%d" % n)
    parity(mask[None], 2, (1.25, 0.5), dist=True, idx=False, tag="long strided sampled n=%d" % n)


def test_long_lines_without_background():
    """Final whole-line passes over samples with and without background."""
    mask = rand_mask((3, 600, 30), 0.002, 600)
    mask[1] = 1
    parity(mask, 2, None, dist=True, idx=False, sq=True, tag="long lines, no background")


def test_sparse_long_envelopes():
    """Few background seeds in a 4-D volume: most first-pass lines are empty."""
    mask = np.ones((2, 12, 20, 24, 28), np.uint8)
    mask[0, 3, 7, 11, 13] = 0
    mask[0, 11, 19, 0, 27] = 0
    mask[1, 0, 0, 0, 0] = 0
    parity(mask, 4, None, dist=True, idx=True, tag="sparse 4-D")
    parity(mask, 4, (1.0, 2.0, 0.5, 1.5), dist=True, idx=True, tag="sparse 4-D sampled")


def test_batch_equals_per_sample():
    mask = workloads.make_mask(3, (24, 20, 36), 4)[:, 0]
    announce("batch vs per-sample")
    whole = run_gpu(mask, 3, None, dist=True, idx=True, sq=True)
    for b in range(mask.shape[0]):
        one = run_gpu(mask[b:b + 1], 3, None, dist=True, idx=True, sq=True)
        for k in ("dist", "idx", "sq"):
            assert np.array_equal(whole[k][b:b + 1], one[k]), (b, k)


def test_deterministic():
    mask = workloads.make_mask(4, (40, 48, 64), 2)
    announce("determinism")
    a = run_gpu(mask, 3, (2.5, 0.8, 0.8), dist=True, idx=True)
    b = run_gpu(mask, 3, (2.5, 0.8, 0.8), dist=True, idx=True)
    assert np.array_equal(a["dist"], b["dist"]) and np.array_equal(a["idx"], b["idx"])


def test_sqrt_is_correctly_rounded():
    """Distances are the correctly rounded float sqrt of the exact squared distance.
    A single zero at the corner of a 1024^2 image gives every sum of two squares up
    to 2 * 1023^2; one at the corner of a 100^3 volume gives every sum of three."""
    for shape in [(1024, 1024), (100, 100, 100)]:
        mask = np.ones((1,) + shape, np.uint8)
        mask[(0,) * (len(shape) + 1)] = 0
        announce("sqrt rounding %s" % (shape,))
        res = run_gpu(mask, len(shape), None, dist=True, sq=True)
        grid = np.indices(shape, dtype=np.int64)
        d2 = sum(g * g for g in grid)
        assert np.array_equal(res["sq"][0], d2)
        assert np.array_equal(res["dist"][0], np.sqrt(d2.astype(np.float64)).astype(np.float32))


# The paired tile takes passes of at least 32768 lines (fewer go to the
# whole-line search), so batches are sized to reach that on every pass.
FUSED = [
    ((513, 65, 64), 2, 0.05),      # final pass reads the mask; 256.5 workgroups (65 rows: past the one-launch small path)
    ((171, 33, 192), 2, 0.01),     # workgroups straddle planes; zeros several words apart
    ((29, 9, 21, 128), 3, 0.2),
    ((103, 5, 160, 64), 3, 0.002), # long lines, mostly empty rows
    ((43, 3, 4, 7, 64), 4, 0.5),
]


@pytest.mark.parametrize("shape,ndim,p_bg", FUSED, ids=["x".join(map(str, s)) for s, _, _ in FUSED])
def test_pass_reading_the_mask(shape, ndim, p_bg):
    """Last extent a multiple of 64: the axis ndim-2 pass computes the
    last-axis distances from the mask itself (checked through the kernel
    names the library reports)."""
    from paper_2608_24738_amd import binding
    mask = rand_mask(shape, p_bg, len(shape) + shape[-1])
    binding.prof_enable(64)
    try:
        parity(mask, ndim, None, dist=True, idx=False, tag="fused")
        names = {n for n, _ in binding.prof_read()}
    finally:
        binding.prof_enable(0)
    assert any(n.startswith("plane_pair") for n in names), names
    assert not any(n.startswith("scan") for n in names), names
    for fill in (0, 1):
        m = np.full(shape, fill, np.uint8)
        m[..., -1, -1] = 1 - fill if fill else 0
        parity(m, ndim, None, dist=True, idx=False, tag="fused fill=%d" % fill)


SEG = [
    ((13, 33, 20, 128), 3, 0.03),    # fused pass hands 16-bit runs to the final pass
    ((22, 6, 10, 4, 64), 4, 0.1),    # axis-1 pass writes 16-bit runs (its input is 32-bit)
    ((9, 5, 6, 7, 128), 4, 0.004),   # a middle pass both reads and writes 16-bit runs
]


@pytest.mark.parametrize("shape,ndim,p_bg", SEG, ids=["x".join(map(str, s)) for s, _, _ in SEG])
def test_half_width_intermediates(shape, ndim, p_bg):
    """Strides that are multiples of 128: consecutive paired passes keep the
    field as 16-bit values in the first half of each 128-element run."""
    from paper_2608_24738_amd import binding
    mask = rand_mask(shape, p_bg, 7 + len(shape))
    binding.prof_enable(64)
    try:
        parity(mask, ndim, None, dist=True, idx=False, tag="half-width")
        names = {n for n, _ in binding.prof_read()}
    finally:
        binding.prof_enable(0)
    assert any(".o16" in n for n in names) and any(".i16" in n for n in names), names
    mask[0] = 1                                   # a sample with no background
    mask[-1] = 0                                  # and one that is all background
    parity(mask, ndim, None, dist=True, idx=False, tag="half-width extremes")


# Last-axis word scan: a wavefront holds 64 / (n / 64) whole lines and its
# stores pass through LDS.  Line lengths 192 and 320 leave idle lanes at the
# end of each wavefront; samples of 3 or 5 lines put several samples in one
# wavefront, so the index slices of its lines are not adjacent in memory.
WORD = [
    ((7, 3, 192), 2, None, True),
    ((11, 5, 320), 2, (1.5, 0.7), True),
    ((4, 5, 3, 192), 3, None, True),
    ((9, 3, 192), 2, None, False),
    ((6, 5, 320), 2, (0.9, 2.0), False),
    ((2, 6, 5, 4096), 2, None, True),
]


@pytest.mark.parametrize("shape,ndim,samp,idx", WORD,
                         ids=["x".join(map(str, s)) + ("-s" if m else "") + ("-i" if i else "")
                              for s, _, m, i in WORD])
def test_word_scan_lanes_and_samples(shape, ndim, samp, idx):
    from paper_2608_24738_amd import binding
    for p_bg, seed in ((0.02, 1), (0.3, 2)):
        mask = rand_mask(shape, p_bg, 100 + seed + len(shape))
        binding.prof_enable(64)
        try:
            parity(mask, ndim, samp, dist=True, idx=idx, tag="word scan p=%g" % p_bg)
            names = {n for n, _ in binding.prof_read()}
        finally:
            binding.prof_enable(0)
        assert any(n.split(".")[0] == "scan_word" for n in names), names
