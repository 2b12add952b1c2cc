"""GPU parity of the mask-reading paired pass when its tile has few rows with
a site, where every element takes the minimum over those rows directly
(sparse backgrounds), and when it has more, where the windowed search runs.
Background fractions are chosen so that tiles fall on both sides of the
limit (8 rows).  Unit euclidean results must equal the oracle's bit for bit,
and so must both chamfer metrics."""
import numpy as np
import pytest

from gpu_util import announce, check_against_oracle, run_gpu
from oracle import edt_oracle

pytestmark = pytest.mark.gpu

# (batch, spatial): the mask-reading pass has >= 32768 lines (paired tile)
SHAPES = [(8, (48, 40, 96)),            # rank 3, axis-1 lines of 40 rows
          (4, (16, 10, 64, 64))]        # rank 4, axis-2 lines of 64 rows
DENSITIES = [2e-4, 1e-3, 2e-3, 5e-3]


def rand_mask(batch, spatial, p_bg, seed):
    rng = np.random.default_rng(seed)
    return (rng.random((batch,) + spatial) >= p_bg).astype(np.uint8)


@pytest.mark.parametrize("p_bg", DENSITIES)
@pytest.mark.parametrize("batch,spatial", SHAPES, ids=["r%d" % len(s) for _, s in SHAPES])
def test_sparse_rows_euclidean(batch, spatial, p_bg):
    from paper_2608_24738_amd import binding
    ndim = len(spatial)
    mask = rand_mask(batch, spatial, p_bg, int(p_bg * 1e6) + ndim)
    announce("direct rows euclidean shape=%s p_bg=%g" % (mask.shape, p_bg))
    binding.prof_enable(64)
    try:
        res = run_gpu(mask, ndim, None, dist=True, idx=False, sq=True)
        names = [n for n, _ in binding.prof_read()]
    finally:
        binding.prof_enable(0)
    assert "plane_pair" in names, names
    ora = edt_oracle.edt(mask, ndim, None, nthreads=16)
    check_against_oracle(mask, ndim, None, res, ora)


@pytest.mark.parametrize("metric", ["taxicab", "chessboard"])
@pytest.mark.parametrize("p_bg", [2e-4, 2e-3])
def test_sparse_rows_chamfer(metric, p_bg):
    import torch
    from paper_2608_24738_amd import binding
    batch, spatial = SHAPES[0]
    mask = rand_mask(batch, spatial, p_bg, 7 + int(p_bg * 1e6))
    announce("direct rows %s shape=%s p_bg=%g" % (metric, mask.shape, p_bg))
    x = torch.from_numpy(mask).to("cuda:0")
    out = torch.empty(mask.shape, dtype=torch.int32, device="cuda:0")
    binding.tm_cdt(x, len(spatial), binding.METRICS[metric], out)
    torch.cuda.synchronize()
    want = edt_oracle.cdt(mask, len(spatial), metric, nthreads=16)
    assert np.array_equal(out.cpu().numpy(), want)
