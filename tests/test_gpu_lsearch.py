"""GPU parity of the whole-line passes (lines longer than the paired 16-bit
tile takes: the windowed search, with the direct minimum where a line
has few sites), at grid sizes around the 32-workgroup sets that the XCD-aware
line-group order permutes: below 32, one full set plus a ragged tail, and
whole sets.  Squared distances and distances must equal the oracle's bit for
bit; the kernel names show that a whole-line pass ran."""
import numpy as np
import pytest

from gpu_util import announce, check_against_oracle, run_gpu
from oracle import edt_oracle

pytestmark = pytest.mark.gpu

# (spatial, batch): axis 0 longer than 256 rows, batch * extent of axis 1 lines
CASES = [((300, 24), 1),      # 3 line groups of 8
         ((300, 264), 1),     # 33 groups: one set of 32 and a tail of 1
         ((520, 200), 2),     # 50 groups
         ((600, 512), 1),     # 64 groups: two whole sets
         ((257, 100), 3)]     # 38 groups, ragged last group


@pytest.mark.parametrize("spatial,batch", CASES, ids=["%dx%d_b%d" % (s[0], s[1], b) for s, b in CASES])
def test_line_search_grids(spatial, batch):
    from paper_2608_24738_amd import binding
    rng = np.random.default_rng(spatial[0] * 1000 + spatial[1] + batch)
    mask = (rng.random((batch,) + spatial) >= 0.003).astype(np.uint8)
    announce("line search shape=%s" % (mask.shape,))
    binding.prof_enable(64)
    try:
        res = run_gpu(mask, 2, None, dist=True, idx=False, sq=True)
        names = [n for n, _ in binding.prof_read()]
    finally:
        binding.prof_enable(0)
    assert any(n.startswith("line_search") for n in names), names
    ora = edt_oracle.edt(mask, 2, None, nthreads=16)
    check_against_oracle(mask, 2, None, res, ora)


# The row scan hands its distances to a whole-line pass of 8 lines per
# workgroup packed to 16 bits (".o16" / ".i16") when every wave's rows pair up
# inside one block of rows (the block's row count a multiple of the wave's
# rows: 4 for 512-wide rows, 8 for 256-wide ones); otherwise as int32.
PACKED_CASES = [((520, 512), 2, True),
                ((514, 512), 1, False),
                ((304, 256), 4, True),
                ((300, 256), 4, False)]


@pytest.mark.parametrize("metric", ["euclidean", "taxicab", "chessboard"])
@pytest.mark.parametrize("spatial,batch,packed", PACKED_CASES,
                         ids=["%dx%d_b%d" % (s[0], s[1], b) for s, b, _ in PACKED_CASES])
def test_packed_row_field(spatial, batch, packed, metric):
    import torch

    from paper_2608_24738_amd import binding
    rng = np.random.default_rng([36, spatial[0], spatial[1], batch])
    mask = (rng.random((batch,) + spatial) >= 0.003).astype(np.uint8)
    mask[0, :, 5] = 0                  # a background column: rows with a zero at 5
    if batch > 1:
        mask[1] = 1                    # one background element: the direct minimum
        mask[1, 7, spatial[1] - 9] = 0
    announce("packed row field %s shape=%s" % (metric, mask.shape))
    binding.prof_enable(64)
    try:
        if metric == "euclidean":
            res = run_gpu(mask, 2, None, dist=True, idx=False, sq=True)
        else:
            x = torch.from_numpy(mask).cuda()
            out = torch.empty(mask.shape, dtype=torch.int32, device=x.device)
            binding.tm_cdt(x, 2, binding.METRICS[metric], out)
            torch.cuda.synchronize()
            got = out.cpu().numpy()
        names = [n for n, _ in binding.prof_read()]
    finally:
        binding.prof_enable(0)
    final = {"euclidean": "line_search_final", "taxicab": "cdt_l1_scan_final",
             "chessboard": "cdt_line_final"}[metric]
    want = ["scan_word.o16", final + ".i16"] if packed else ["scan_word", final]
    assert list(dict.fromkeys(names)) == want, names     # run_gpu makes two calls
    if metric == "euclidean":
        check_against_oracle(mask, 2, None, res, edt_oracle.edt(mask, 2, None, nthreads=16))
    else:
        assert np.array_equal(got, edt_oracle.cdt(mask, 2, metric, nthreads=16))


@pytest.mark.parametrize("metric", ["euclidean", "taxicab", "chessboard"])
def test_packed_row_field_3d(metric):
    # 2 x 4 x 600 x 256: the row scan (32-position words, 8 rows per wave)
    # packs for the axis-1 whole-line pass, which is not the last one
    import torch

    from paper_2608_24738_amd import binding
    rng = np.random.default_rng(37)
    mask = (rng.random((2, 4, 600, 256)) >= 0.002).astype(np.uint8)
    mask[1, 2] = 1                     # a plane without background
    announce("packed row field 3-D %s shape=%s" % (metric, mask.shape))
    binding.prof_enable(64)
    try:
        if metric == "euclidean":
            res = run_gpu(mask, 3, None, dist=True, idx=False, sq=True)
        else:
            x = torch.from_numpy(mask).cuda()
            out = torch.empty(mask.shape, dtype=torch.int32, device=x.device)
            binding.tm_cdt(x, 3, binding.METRICS[metric], out)
            torch.cuda.synchronize()
            got = out.cpu().numpy()
        names = list(dict.fromkeys(n for n, _ in binding.prof_read()))
    finally:
        binding.prof_enable(0)
    middle = {"euclidean": "line_search.i16", "taxicab": "cdt_l1_scan.i16", "chessboard": "cdt_line.i16"}[metric]
    assert names[:2] == ["scan_word.o16", middle], names
    if metric == "euclidean":
        check_against_oracle(mask, 3, None, res, edt_oracle.edt(mask, 3, None, nthreads=16))
    else:
        assert np.array_equal(got, edt_oracle.cdt(mask, 3, metric, nthreads=16))
