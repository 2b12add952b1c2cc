"""GPU parity of the plane-ordered signed transform (rank 3, 128 x 128
planes, n0 <= 128: k_col_scan_signed then k_plane_signed) against the
oracle's EDT(M) - EDT(not M), bit-exact, on Bernoulli masks of several
densities, balls, columns and planes of one class, single-class samples
(the virtual element), axis-0 extents 1 .. 128, and on the inputs that
leave the plane path (misaligned mask, n0 above 128, other plane sizes)."""
import numpy as np
import pytest

from gpu_util import announce
from oracle import edt_oracle
from paper_2608_24738_amd import workloads

pytestmark = pytest.mark.gpu

PLANE_KERNELS = ["col_scan_signed", "plane_signed_final"]


def run_signed(x, ndim):
    """Signed transform of the device mask x; returns (result, kernel names)."""
    import torch
    from paper_2608_24738_amd import binding
    out = torch.empty(x.shape, dtype=torch.float32, device=x.device)
    binding.prof_enable(64)
    try:
        binding.tm_edt_signed(x, ndim, out)
        torch.cuda.synchronize()
        names = [n for n, _ in binding.prof_read()]
    finally:
        binding.prof_enable(0)
    return out.cpu().numpy(), names


def check(mask, tag, plane=True):
    import torch
    announce("psigned %s shape=%s" % (tag, mask.shape))
    x = torch.from_numpy(np.ascontiguousarray(mask)).to("cuda:0")
    got, names = run_signed(x, 3)
    if plane:
        assert names == PLANE_KERNELS, names
    else:
        assert "plane_signed_final" not in names, names
    want = edt_oracle.signed_edt(mask, 3, nthreads=8)
    if not np.array_equal(got, want):
        bad = np.argwhere(got != want)
        k = tuple(bad[0])
        raise AssertionError("%s %s: %d elements differ; first at %s: got %r want %r"
                             % (tag, mask.shape, len(bad), k, got[k], want[k]))


def bern(shape, p_fg, seed):
    rng = np.random.default_rng(seed)
    return (rng.random(shape) < p_fg).astype(np.uint8)


CASES = [
    (1, 1, 0.5), (1, 2, 0.5), (2, 16, 0.9), (1, 17, 0.1), (3, 33, 0.97),
    (1, 100, 0.5), (1, 128, 0.995), (2, 128, 0.03),
]


@pytest.mark.parametrize("batch,n0,p", CASES, ids=["b%d-n%d-p%g" % c for c in CASES])
def test_bernoulli(batch, n0, p):
    check(bern((batch, n0, 128, 128), p, 900 + n0), "bernoulli p=%g" % p)


def test_balls():
    w = workloads.WORKLOADS[3]
    mask = workloads.make_mask(3, (w.spatial[0] // 2,) + tuple(w.spatial[1:]), 2)[:, 0]
    check(mask, "balls")


def test_one_class_structures():
    # a sample of one class (both classes), a plane of one class, columns
    # along axis 0 of one class, a single element of the other class
    m = bern((5, 40, 128, 128), 0.6, 11)
    m[0] = 1
    m[1] = 0
    m[2, 7] = 0
    m[2, 9] = 1
    m[3, :, 5, :] = 1
    m[3, :, :, 77] = 0
    m[4] = 1
    m[4, 39, 127, 0] = 0
    check(m, "one-class structures")


def test_far_corners():
    # the longest distances the plane path meets: one element of the other
    # class in a corner of a 128^3 sample, each way round
    m = np.ones((2, 128, 128, 128), np.uint8)
    m[0, 0, 0, 0] = 0
    m[1] = 0
    m[1, 127, 127, 127] = 1
    check(m, "far corners")


def test_full_workload():
    mask = workloads.make_mask(3)[:, 0]
    check(mask, "8x128^3")


def test_paths_beside_the_plane():
    import torch
    # n0 above 128 and 64 x 64 planes take the whole-line passes
    check(bern((1, 130, 128, 128), 0.5, 5), "n0=130", plane=False)
    check(bern((2, 20, 64, 64), 0.5, 6), "64x64", plane=False)
    # a mask at an odd address: same result through the other path
    mask = bern((1, 9, 128, 128), 0.7, 7)
    buf = torch.zeros(mask.size + 1, dtype=torch.uint8, device="cuda:0")
    x = buf[1:].view(mask.shape)
    x.copy_(torch.from_numpy(mask).to("cuda:0"))
    got, names = run_signed(x, 3)
    assert "plane_signed_final" not in names, names
    assert np.array_equal(got, edt_oracle.signed_edt(mask, 3, nthreads=8))
