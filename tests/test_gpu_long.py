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
    # sampled, distances only: the flat-index carrier inside out_dist
    ((12000, 3), 2, 1e-3, (1.5, 1.0), False, "fh_index_final"),
    ((20000, 2), 1, 5e-4, (0.7, 2.0), False, "fh_index_final"),
    ((30000, 3), 1, 1e-3, None, True, "fh_index_final"),           # index carrier
    ((30000, 3), 1, 1e-3, (1.5, 1.0), True, "fh_index_final"),
    # past every LDS-resident kernel: the envelope in the line's own storage
    ((70000, 3), 1, 1e-3, (1.5, 1.0), False, "fh_long_final"),     # carrier inside out_dist
    ((70000, 3), 1, 1e-3, (1.5, 1.0), True, "fh_long_final"),
    ((70000, 3), 1, 3e-2, (0.8, 2.5), True, "fh_long_final"),      # dense: many envelope entries
    ((70000, 3), 1, 1e-3, None, False, "fh_long_final"),           # squared distances past 2^31
    ((70000, 3), 1, 1e-3, None, True, "fh_long_final"),
    ((45000, 3), 2, 1e-3, None, False, "fh_long_final"),           # tm_edt_sq through the carrier
    ((45000, 3), 1, 5e-2, None, True, "fh_long_final"),
    ((3, 45000, 2), 1, 1e-3, None, False, "fh_long"),              # long middle axis
    ((2, 50000, 3), 1, 1e-3, (2.0, 0.5, 1.0), True, "fh_long"),
]


@pytest.mark.parametrize("spatial,batch,p_bg,sampling,want_idx,kernel", CASES,
                         ids=["%s-b%d%s%s" % ("x".join(map(str, c[0])), c[1], "-samp" if c[3] else "",
                                              "-idx" if c[4] else "") for c in CASES])
def test_long_strided_lines(spatial, batch, p_bg, sampling, want_idx, kernel):
    mask = sparse_mask(spatial, batch, p_bg, len(spatial) * 100 + spatial[0] % 97)
    nd = len(spatial)
    unit = sampling is None
    # exact squared distances need sum(n^2) < 2^31 (tm_edt_sq's int32 output)
    sq = unit and sum(int(n) ** 2 for n in spatial) < 2 ** 31 - 1
    announce("long lines %s batch=%d sampling=%s idx=%s sq=%s" % (spatial, batch, sampling, want_idx, sq))
    res, names = run_named(mask, nd, sampling, dist=True, idx=want_idx, sq=sq)
    assert kernel in names, names
    check_against_oracle(mask, nd, sampling, res, oracle(mask, nd, sampling))
    if sq:
        # tm_edt_sq with indices: the squared distances and coordinates
        # written by the same final pass
        announce("long lines %s: tm_edt_sq with indices" % (spatial,))
        res2, _ = run_named(mask, nd, None, dist=False, idx=True, sq=True)
        ora = oracle(mask, nd)
        assert np.array_equal(res2["sq"], ora["sq"])


def test_long_line_without_background():
    """A sample with no background at all along a long strided axis: the
    virtual element (-1, 0) in the final envelope pass."""
    mask = np.ones((1, 15000, 2), np.uint8)
    announce("long line, no background, (15000, 2)")
    res, names = run_named(mask, 2, None, dist=True, idx=True, sq=True)
    check_against_oracle(mask, 2, None, res, oracle(mask, 2))


def test_long_line_without_background_sampled():
    """No background along a line too long for LDS: the virtual element in
    the envelope kernel that keeps its stack in the line."""
    mask = np.ones((1, 50000, 2), np.uint8)
    samp = (2.0, 1.0)
    announce("long line, no background, (50000, 2), sampled, with indices")
    res, names = run_named(mask, 2, samp, dist=True, idx=True)
    assert "fh_long_final" in names, names
    check_against_oracle(mask, 2, samp, res, oracle(mask, 2, samp))


def test_very_long_rank1_line():
    """One 1-D line of 50 million elements (more 1024-element chunks than a
    per-chunk table in LDS would hold): the last-axis scan parks its carries
    in the output.  Squared distances reach 2.5e15, so only tm_edt applies."""
    n = 50_000_000
    rng = np.random.default_rng([11, 7])
    mask = np.ones((1, n), np.uint8)
    mask[0, rng.integers(0, n, 40)] = 0
    mask[0, :3] = 1
    announce("rank-1 line of %d elements, dist + idx" % n)
    res, names = run_named(mask, 1, None, dist=True, idx=True, sq=False)
    assert "scan_long" in names, names
    # nearest zero from the sorted zero positions (the left one on ties):
    # the textbook 1-D transform, at a size the oracle's line sweep is slow for
    z = np.flatnonzero(mask[0] == 0)
    x = np.arange(n, dtype=np.int64)
    k = np.searchsorted(z, x)
    left = np.where(k > 0, z[np.maximum(k - 1, 0)], -(1 << 40))
    right = np.where(k < len(z), z[np.minimum(k, len(z) - 1)], 1 << 40)
    near = np.where(x - left <= right - x, left, right)
    d2 = (x - near) ** 2
    assert np.array_equal(res["idx"].reshape(-1), near)
    assert np.array_equal(res["dist"][0], np.sqrt(d2.astype(np.float64)).astype(np.float32))


def test_long_signed_and_chamfer_lines():
    """The signed transform and the chamfer transforms along 30 000- to
    70 000-element strided lines (whole lines in LDS, one or two per
    workgroup; taxicab lines of any length by two running minima)."""
    import torch
    from paper_2608_24738_amd import binding
    dev = torch.device("cuda:0")
    mask = sparse_mask((30000, 3), 1, 2e-3, 5)
    mask[0, 20000:21000] = 0                                     # a run of background
    x = torch.from_numpy(mask).to(dev)
    announce("signed transform (30000, 3)")
    out = torch.empty(mask.shape, dtype=torch.float32, device=dev)
    binding.prof_enable(64)
    try:
        binding.tm_edt_signed(x, 2, out)
        torch.cuda.synchronize()
        names = {n for n, _ in binding.prof_read()}
    finally:
        binding.prof_enable(0)
    assert "line_search_signed_final" in names, names
    assert np.array_equal(out.cpu().numpy(), edt_oracle.signed_edt(mask, 2))
    for spatial, metric, kernel in [((30000, 3), "taxicab", "cdt_line_final"),
                                    ((30000, 3), "chessboard", "cdt_line_final"),
                                    ((50000, 3), "chessboard", "cdt_line_final"),
                                    ((70000, 3), "taxicab", "cdt_l1_long_final")]:
        m = sparse_mask(spatial, 1, 1e-3, spatial[0] % 89)
        announce("chamfer %s %s" % (metric, spatial))
        xm = torch.from_numpy(m).to(dev)
        o = torch.empty(m.shape, dtype=torch.int32, device=dev)
        binding.prof_enable(64)
        try:
            binding.tm_cdt(xm, 2, binding.METRICS[metric], o)
            torch.cuda.synchronize()
            names = {n for n, _ in binding.prof_read()}
        finally:
            binding.prof_enable(0)
        assert kernel in names, (metric, spatial, names)
        assert np.array_equal(o.cpu().numpy(), edt_oracle.cdt(m, 2, metric)), (metric, spatial)
    # no background at all along a long taxicab line: -1 everywhere
    m = np.ones((1, 70000, 2), np.uint8)
    announce("chamfer taxicab (70000, 2) without background")
    o = torch.empty(m.shape, dtype=torch.int32, device=dev)
    binding.tm_cdt(torch.from_numpy(m).to(dev), 2, binding.METRICS["taxicab"], o)
    torch.cuda.synchronize()
    assert (o.cpu().numpy() == -1).all()
