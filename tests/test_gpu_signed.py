"""GPU parity of the signed transform (tm_edt_signed) against the oracle's
EDT(M) - EDT(not M), bit-exact (both sides round the square root of the
same exact integer, with the class sign), on shapes that run every kernel
path: the register and the long first-pass scans, rank 1, the whole-line
search with 8 and 4 lines per workgroup, single-class samples."""
import numpy as np
import pytest

from gpu_util import announce
from oracle import edt_oracle
from paper_2608_24738_amd import workloads

pytestmark = pytest.mark.gpu


def rand_mask(shape, p_bg, seed):
    rng = np.random.default_rng(seed)
    return (rng.random(shape) >= p_bg).astype(np.uint8)


def run_signed(mask, ndim):
    import torch
    from paper_2608_24738_amd import binding
    x = torch.from_numpy(np.ascontiguousarray(mask)).to("cuda:0")
    out = torch.empty(mask.shape, dtype=torch.float32, device="cuda:0")
    binding.tm_edt_signed(x, ndim, out)
    torch.cuda.synchronize()
    return out.cpu().numpy()


def check(mask, ndim, tag=""):
    announce("signed %s shape=%s" % (tag, mask.shape))
    got = run_signed(mask, ndim)
    want = edt_oracle.signed_edt(mask, ndim, nthreads=8)
    if not np.array_equal(got, want):
        bad = np.argwhere(got != want)
        k = tuple(bad[0])
        raise AssertionError("%s %s: %d elements differ; first at %s: got %r want %r"
                             % (tag, mask.shape, len(bad), k, got[k], want[k]))


SHAPES = [
    (3, (1,), 0.5),
    (2, (37,), 0.3),                 # rank 1
    (2, (1500,), 0.01),              # rank 1, long first-pass scan
    (2, (70, 45), 0.2),
    (2, (64, 1024), 0.02),           # 16 register chunks
    (2, (5, 1500), 0.01),            # long first-pass scan feeding a strided pass
    (2, (300, 40), 0.05),
    (2, (20, 16, 128), 0.1),
    (1, (9, 33, 17), 0.5),
    (1, (5, 6, 7, 8), 0.3),
    (1, (2, 2, 2, 2, 2, 2, 2, 3), 0.4),
    (1, (6000, 3), 0.001),           # 4 lines per workgroup
    (2, (1, 1), 0.5),
    (1, (50, 1), 0.1),
]


@pytest.mark.parametrize("batch,spatial,p", SHAPES,
                         ids=["b%d-%s" % (b, "x".join(map(str, s))) for b, s, _ in SHAPES])
def test_parity(batch, spatial, p):
    mask = rand_mask((batch,) + spatial, p, 500 + sum(spatial))
    check(mask, len(spatial), "shape")


def test_one_class_samples():
    mask = rand_mask((4, 30, 40), 0.1, 3)
    mask[1] = 1
    mask[2] = 0
    check(mask, 2, "one class")
    m1 = np.ones((2, 700), np.uint8)
    m1[1] = 0
    check(m1, 1, "one class rank 1")


@pytest.mark.parametrize("key", (3, 10))
def test_workload_full_size(key):
    w = workloads.WORKLOADS[key]
    mask = workloads.make_mask(key)[:, 0]
    check(mask, w.ndim, "full %s" % w.name)


def test_batch_equals_per_sample():
    mask = workloads.make_mask(3, (24, 20, 36), 3)[:, 0]
    whole = run_signed(mask, 3)
    for b in range(3):
        assert np.array_equal(run_signed(mask[b:b + 1], 3), whole[b:b + 1])
