"""Long strided lines (paper, Section 2.3.2: lines too long for on-chip
memory): parity with the oracle, element by element, for lines from about
10 000 to the longest the interface takes, through tm_edt and tm_edt_sq,
with and without indices, unit and sampled, and the kernel each case runs.
"""
import numpy as np
import pytest

from gpu_util import announce, check_against_oracle, run_gpu
from oracle import edt_oracle

pytestmark = pytest.mark.gpu


def oracle(mask, ndim, sampling=None):
    return edt_oracle.edt(mask, ndim, sampling, nthreads=16)


def sparse_mask(spatial, batch, p_bg, seed):
    rng = np.random.default_rng([11, seed])
    m = (rng.random((batch,) + tuple(spatial)) >= p_bg).astype(np.uint8)
    # a stretch of background rows near one end, a long empty run elsewhere
    m[:, 1:3] = 0
    return m


def run_named(mask, ndim, sampling=None, dist=True, idx=False, sq=False):
    from paper_2608_24738_amd import binding
    binding.prof_enable(64)
    try:
        res = run_gpu(mask, ndim, sampling, dist=dist, idx=idx, sq=sq)
        names = {n for n, _ in binding.prof_read()}
    finally:
        binding.prof_enable(0)
    return res, names


# (spatial, batch, p_bg, sampling, index output, kernel expected on axis 0)
CASES = [
    ((12000, 3), 2, 1e-3, None, False, "fh_field_final"),          # packed stack entries
    ((20000, 2), 1, 5e-4, None, False, "fh_field_final"),          # packed, two lines per workgroup
    ((12000, 600), 1, 2e-4, None, False, "fh_field_final"),        # apex + value need 33 bits: unpacked
    ((12000, 3), 2, 1e-3, (1.5, 1.0), False, "fh_field_final"),    # sampled: double breakpoints
    ((20000, 2), 1, 5e-4, (0.7, 2.0), False, "fh_field_final"),
    ((30000, 3), 1, 1e-3, None, True, "fh_index_final"),           # index carrier
    ((30000, 3), 1, 1e-3, (1.5, 1.0), True, "fh_index_final"),
]


@pytest.mark.parametrize("spatial,batch,p_bg,sampling,want_idx,kernel", CASES,
                         ids=["%s-b%d%s%s" % ("x".join(map(str, c[0])), c[1], "-samp" if c[3] else "",
                                              "-idx" if c[4] else "") for c in CASES])
def test_long_strided_lines(spatial, batch, p_bg, sampling, want_idx, kernel):
    mask = sparse_mask(spatial, batch, p_bg, len(spatial) * 100 + spatial[0] % 97)
    nd = len(spatial)
    unit = sampling is None
    announce("long lines %s batch=%d sampling=%s idx=%s" % (spatial, batch, sampling, want_idx))
    res, names = run_named(mask, nd, sampling, dist=True, idx=want_idx, sq=unit)
    assert kernel in names, names
    check_against_oracle(mask, nd, sampling, res, oracle(mask, nd, sampling))


def test_long_line_without_background():
    """A sample with no background at all along a long strided axis: the
    virtual element (-1, 0) in the final envelope pass."""
    mask = np.ones((1, 15000, 2), np.uint8)
    announce("long line, no background, (15000, 2)")
    res, names = run_named(mask, 2, None, dist=True, idx=True, sq=True)
    check_against_oracle(mask, 2, None, res, oracle(mask, 2))
