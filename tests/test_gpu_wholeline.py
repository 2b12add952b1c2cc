"""GPU parity of the whole-line pass (unit sampling, distances only): lines
from two rows to a few thousand, ragged workgroups, lines without any site,
lines of 512 rows and more with one or a few sites (the direct minimum over
the occupied rows, taken when every line of a workgroup has at most 32),
workgroups mixing such lines with denser ones, equidistant sites.
Every squared distance and distance must equal the oracle's."""
import numpy as np
import pytest

from gpu_util import announce, check_against_oracle, run_gpu
from oracle import edt_oracle

pytestmark = pytest.mark.gpu


def run_named(mask, ndim):
    from paper_2608_24738_amd import binding
    binding.prof_enable(64)
    try:
        res = run_gpu(mask, ndim, None, dist=True, idx=False, sq=True)
        names = {n for n, _ in binding.prof_read()}
    finally:
        binding.prof_enable(0)
    return res, names


# (spatial, batch, background density)
CASES = [
    ((300, 7), 2, 0.01),        # short lines: the search only
    ((512, 64), 1, 0.003),      # the 2-D 512^2 length
    ((1024, 40), 1, 0.001),
    ((2000, 9), 1, 0.02),       # about 40 sites per line: windowed search
    ((17, 300), 3, 0.05),       # below the paired tile's line count
    ((700, 130), 1, 0.2),       # dense
    ((260, 260, 3), 1, 0.002),  # middle axis and final axis both whole-line
]


@pytest.mark.parametrize("spatial,batch,p_bg", CASES,
                         ids=["%s-b%d" % ("x".join(map(str, c[0])), c[1]) for c in CASES])
def test_wholeline_parity(spatial, batch, p_bg):
    rng = np.random.default_rng([13, spatial[0], spatial[1], batch])
    mask = (rng.random((batch,) + tuple(spatial)) >= p_bg).astype(np.uint8)
    nd = len(spatial)
    announce("whole-line parity %s batch=%d p_bg=%g" % (spatial, batch, p_bg))
    res, names = run_named(mask, nd)
    assert any(n.startswith("line_search") for n in names), names
    check_against_oracle(mask, nd, None, res, edt_oracle.edt(mask, nd, None, nthreads=16))


def test_wholeline_single_site_and_empty_lines():
    """Columns with one background element each (one chunk sweeps the whole
    line), columns with none (no site: the next pass or the virtual element),
    and a sample without any background."""
    n0, n1 = 1024, 37
    mask = np.ones((3, n0, n1), np.uint8)
    rng = np.random.default_rng(5)
    for c in range(0, n1, 2):
        mask[0, rng.integers(0, n0), c] = 0
    mask[1, 0, 5] = 0
    mask[1, n0 - 1, 30] = 0
    announce("whole-line single sites / empty lines (3, %d, %d)" % (n0, n1))
    res, names = run_named(mask, 2)
    assert any(n.startswith("line_search") for n in names), names
    check_against_oracle(mask, 2, None, res, edt_oracle.edt(mask, 2, None, nthreads=16))


def test_wholeline_ties_and_equal_values():
    """Many equal values and equidistant sites (breakpoints exactly on
    integers): the exact comparisons must still give the minimum."""
    n0 = 640
    mask = np.ones((2, n0, 64), np.uint8)
    mask[0, ::8, :] = 0                  # equidistant background rows
    mask[0, :, ::16] = 0
    mask[1, ::33, ::7] = 0
    announce("whole-line ties (2, %d, 64)" % n0)
    res, names = run_named(mask, 2)
    assert any(n.startswith("line_search") for n in names), names
    check_against_oracle(mask, 2, None, res, edt_oracle.edt(mask, 2, None, nthreads=16))


@pytest.mark.parametrize("count", [1, 31, 32, 33])
def test_wholeline_site_counts(count):
    """Columns of 768 rows whose background rows number exactly `count` (the
    direct minimum up to 32 sites per line, the search above), plus a
    workgroup whose lines differ (one line with 200 sites)."""
    n0, n1 = 768, 24
    rng = np.random.default_rng([17, count])
    mask = np.ones((2, n0, n1), np.uint8)
    for b in range(2):
        for c in range(n1):
            mask[b, rng.choice(n0, count, replace=False), c] = 0
    mask[1, rng.choice(n0, 200, replace=False), 3] = 0   # a dense column among sparse ones
    # (the first pass is along the rows, so a column's sites are the rows
    # holding any background; keep each background row within one column)
    announce("whole-line site counts %d, (2, %d, %d)" % (count, n0, n1))
    res, names = run_named(mask, 2)
    assert any(n.startswith("line_search") for n in names), names
    check_against_oracle(mask, 2, None, res, edt_oracle.edt(mask, 2, None, nthreads=16))
