"""GPU parity of the chamfer transforms (tm_cdt) against the chamfer oracle,
element by element and bit-exact (int32 distances, -1 for samples without
background), on shapes chosen to run every kernel path: the last-axis scan
(word, span and long variants), the paired tile with and without the
mask-reading first pass and the 16-bit hand-over, the whole-line LDS pass
for long lines or values past 16 bits, and rank 1.  At the full workload
sizes the result is checked against the chamfer equations everywhere plus
brute-force spot checks."""
import numpy as np
import pytest

from gpu_util import announce
from invariants import chamfer_fixed_point_violations
from oracle import edt_oracle
from paper_2608_24738_amd import workloads

pytestmark = pytest.mark.gpu

CHAMFER = ("taxicab", "chessboard")


def rand_mask(shape, p_bg, seed):
    rng = np.random.default_rng(seed)
    return (rng.random(shape) >= p_bg).astype(np.uint8)


def run_cdt(mask, ndim, metric, stream=None):
    import torch
    from paper_2608_24738_amd import binding
    dev = torch.device("cuda:0")
    x = torch.from_numpy(np.ascontiguousarray(mask)).to(dev)
    out = torch.empty(mask.shape, dtype=torch.int32, device=dev)
    binding.tm_cdt(x, ndim, binding.METRICS[metric], out, stream=stream)
    torch.cuda.synchronize()
    return out.cpu().numpy()


def check(mask, ndim, metric, tag=""):
    announce("cdt %s %s shape=%s" % (tag, metric, mask.shape))
    got = run_cdt(mask, ndim, metric)
    want = edt_oracle.cdt(mask, ndim, metric, nthreads=8)
    if not np.array_equal(got, want):
        bad = np.argwhere(got != want)
        k = tuple(bad[0])
        raise AssertionError("%s %s %s: %d elements differ; first at %s: got %d want %d"
                             % (tag, metric, mask.shape, len(bad), k, got[k], want[k]))


# (batch, spatial, background fraction).  Passes of fewer than 32768 lines
# take the whole-line search; larger batches below take the paired tile.
SHAPES = [
    (3, (1,), 0.0),                 # rank 1, one element, no background
    (2, (37,), 0.1),                # rank 1, span scan
    (4, (128,), 0.03),              # rank 1, word scan
    (2, (1500,), 0.002),            # rank 1, long scan
    (2, (70, 45), 0.02),            # odd last extent
    (2, (100, 64), 0.02),
    (3, (256, 256), 0.001),
    (1, (200, 96), 0.01),
    (2, (129, 33), 0.05),
    (2, (20, 16, 128), 0.002),
    (2, (9, 33, 17), 0.03),
    (1, (300, 5), 0.01),
    (2, (600, 40, 3), 0.003),
    (1, (3, 400, 8), 0.002),
    (1, (5, 6, 7, 8), 0.01),
    (2, (3, 4, 3, 4, 5), 0.02),
    (1, (2, 2, 2, 2, 2, 2, 2, 3), 0.05),
    (2, (1, 1), 0.0),
    (1, (1, 50), 0.05),
    (1, (50, 1), 0.05),
]

# Batches large enough for the paired tile on every strided pass, with the
# kernel names it must report: the mask-reading first pass, 16-row blocks
# past 8, and the 16-bit hand-over between paired passes.
PAIRED = [
    (513, (50, 64), 0.02, ("cdt_plane_final",)),
    (1000, (129, 33), 0.05, ("cdt_pair_final",)),
    (13, (33, 20, 128), 0.005, ("cdt_plane.o16", "cdt_pair_final.i16")),
    (43, (3, 4, 7, 64), 0.1, ("cdt_plane", "cdt_pair", "cdt_pair_final")),
    (60, (600, 40, 3), 0.003, ("cdt_pair", "cdt_line_final")),
]


@pytest.mark.parametrize("metric", CHAMFER)
@pytest.mark.parametrize("batch,spatial,p", SHAPES,
                         ids=["b%d-%s" % (b, "x".join(map(str, s))) for b, s, _ in SHAPES])
def test_parity(metric, batch, spatial, p):
    mask = rand_mask((batch, 1) + spatial, p, 1000 * len(spatial) + sum(spatial))
    check(mask, len(spatial), metric, "shape")


@pytest.mark.parametrize("metric", CHAMFER)
@pytest.mark.parametrize("batch,spatial,p,kernels", PAIRED,
                         ids=["b%d-%s" % (b, "x".join(map(str, s))) for b, s, _, _ in PAIRED])
def test_paired_tile(metric, batch, spatial, p, kernels):
    from paper_2608_24738_amd import binding
    mask = rand_mask((batch, 1) + spatial, p, 77 + sum(spatial))
    mask[0] = 1                                   # a sample without background
    binding.prof_enable(64)
    try:
        check(mask, len(spatial), metric, "paired")
        names = {n for n, _ in binding.prof_read()}
    finally:
        binding.prof_enable(0)
    for k in kernels:
        if metric == "taxicab" and k == "cdt_line_final":
            k = "cdt_l1_scan_final"          # taxicab lines: prefix and suffix minima
        assert k in names, (k, names)


@pytest.mark.parametrize("metric", CHAMFER)
def test_values_past_16_bits(metric):
    # a 70000-long last axis: values reach past 65535, so the short lines of
    # axis 0 go through the whole-line pass
    mask = np.ones((2, 1, 5, 70000), np.uint8)
    mask[0, 0, 1, 3] = 0
    mask[0, 0, 4, 69000] = 0
    mask[1, 0, 2, 35000] = 0
    check(mask, 2, metric, "wide")


@pytest.mark.parametrize("metric", CHAMFER)
@pytest.mark.parametrize("n", [1300, 4000, 12000])
def test_long_lines(metric, n):
    # whole-line search with 8 and (n = 12000) 4 lines per workgroup (16-bit
    # tile), one sample without background
    mask = rand_mask((2, 1, n, 3), 0.004, n)
    mask[1] = 1
    check(mask, 2, metric, "long")


@pytest.mark.parametrize("metric", CHAMFER)
def test_long_lines_past_16_bits(metric):
    # 32-bit tile: a 65600-long last axis and 640-long strided lines
    mask = np.ones((1, 1, 640, 65600), np.uint8)
    for y, x in ((3, 5), (600, 65000), (320, 30000), (639, 0)):
        mask[0, 0, y, x] = 0
    check(mask, 2, metric, "long wide")


@pytest.mark.parametrize("metric", CHAMFER)
def test_mixed_batch_without_background(metric):
    mask = rand_mask((5, 1, 40, 64), 0.01, 11)
    mask[1] = 1
    mask[3] = 1
    mask[4] = 0
    check(mask, 2, metric, "mixed")
    got = run_cdt(mask, 2, metric)
    assert np.all(got[1] == -1) and np.all(got[3] == -1) and np.all(got[4] == 0)


@pytest.mark.parametrize("metric", CHAMFER)
def test_batch_equals_per_sample_and_deterministic(metric):
    mask = workloads.make_mask(8, (96, 160), 4)
    whole = run_cdt(mask, 2, metric)
    for b in range(4):
        assert np.array_equal(run_cdt(mask[b:b + 1], 2, metric), whole[b:b + 1])
    assert np.array_equal(run_cdt(mask, 2, metric), whole)


@pytest.mark.parametrize("metric", CHAMFER)
@pytest.mark.parametrize("key", (7, 8))
def test_workload_full_size(key, metric):
    # the configuration the benchmark times; brute force over every element
    # is too slow here, so: the chamfer equations at every element (they fix
    # the result uniquely) and brute-force values at 512 seeded points
    w = workloads.WORKLOADS[key]
    mask = workloads.make_mask(key)
    announce("cdt full %s %s" % (w.name, metric))
    got = run_cdt(mask, w.ndim, metric)
    rng = np.random.default_rng([key, 5])
    for b in range(w.batch):
        assert chamfer_fixed_point_violations(mask[b, 0], got[b, 0], metric) == 0, b
        pts = np.stack([rng.integers(0, n, 64) for n in w.spatial], axis=1)
        ref = edt_oracle.metric_dt_at(mask[b, 0], metric, pts)
        assert np.array_equal(got[b, 0][tuple(pts.T)], ref.astype(np.int64)), b


def test_twin_of_the_workloads():
    for key in (7, 8):
        mask = workloads.make_mask(key, (150, 130), 3)
        for metric in CHAMFER:
            check(mask, 2, metric, "twin%d" % key)


def test_rejects_euclidean_and_unknown_metrics():
    import torch
    from paper_2608_24738_amd import binding
    x = torch.ones((1, 1, 8, 8), dtype=torch.uint8, device="cuda:0")
    out = torch.empty((1, 1, 8, 8), dtype=torch.int32, device="cuda:0")
    for code in (0, 3):
        with pytest.raises(binding.TMError):
            binding.tm_cdt(x, 2, code, out)


@pytest.mark.parametrize("metric", ["chessboard"])
def test_ordered_column_pass(metric):
    """tm_cdt_ws (chessboard): the column pass of 8 x 1024^2 discs dispatched heaviest
    first from the row scan's estimates (units of four 8-column workgroups):
    equal to tm_cdt, the chamfer equations at every element and brute-force
    values at seeded points (as the full-size test), counters cleared, the
    order a permutation."""
    import torch
    from paper_2608_24738_amd import binding
    dev = torch.device("cuda:0")
    mask = workloads.make_mask(7)[:, 0].copy()
    mask[5] = 1                                     # a sample without background: -1
    announce("cdt ordered %s shape=%s" % (metric, mask.shape))
    code = binding.METRICS[metric]
    need = binding.tm_cdt_workspace_size(2, mask.shape[1:], mask.shape[0], code)
    assert need > 0
    x = torch.from_numpy(mask).to(dev)
    ws = torch.zeros(need // 4, dtype=torch.int32, device=dev)
    out = torch.empty(mask.shape, dtype=torch.int32, device=dev)
    binding.prof_enable(64)
    try:
        binding.tm_cdt_ws(x, 2, code, out, ws)
        torch.cuda.synchronize()
        names = [n for n, _ in binding.prof_read()]
    finally:
        binding.prof_enable(0)
    assert names == ["scan_word.cost.o16", "order", "cdt_line_final.i16"], names
    got = out.cpu().numpy()
    assert np.array_equal(got, run_cdt(mask, 2, metric))
    assert (got[5] == -1).all()
    rng = np.random.default_rng([7, 6])
    for b in range(mask.shape[0]):
        if b == 5:
            continue
        assert chamfer_fixed_point_violations(mask[b], got[b], metric) == 0, b
        pts = np.stack([rng.integers(0, n, 64) for n in mask.shape[1:]], axis=1)
        ref = edt_oracle.metric_dt_at(mask[b], metric, pts)
        assert np.array_equal(got[b][tuple(pts.T)], ref.astype(np.int64)), b
    w = ws.cpu().numpy()
    units = need // 8
    assert not w[:units].any()
    assert np.array_equal(np.sort(w[units:2 * units]), np.arange(units))


def full_size_checks(mask, got, metric, key):
    """The chamfer equations at every element and brute-force values at 64
    seeded points per sample (the full-size pattern); -1 on samples without
    background."""
    rng = np.random.default_rng([key, 6])
    for b in range(mask.shape[0]):
        if not (mask[b] == 0).any():
            assert (got[b] == -1).all(), b
            continue
        assert chamfer_fixed_point_violations(mask[b], got[b], metric) == 0, b
        pts = np.stack([rng.integers(0, n, 64) for n in mask.shape[1:]], axis=1)
        ref = edt_oracle.metric_dt_at(mask[b], metric, pts)
        assert np.array_equal(got[b][tuple(pts.T)], ref.astype(np.int64)), b


def test_taxicab_scan_full_workload():
    """8 x 1024^2 discs, taxicab, through tm_cdt_ws: the row scan packs its
    distances and the column pass is the prefix / suffix minimum (even work
    per group: no workspace, no order)."""
    import torch
    from paper_2608_24738_amd import binding
    mask = workloads.make_mask(7)[:, 0].copy()
    mask[5] = 1
    announce("taxicab scan shape=%s" % (mask.shape,))
    code = binding.METRICS["taxicab"]
    assert binding.tm_cdt_workspace_size(2, mask.shape[1:], mask.shape[0], code) == 0
    x = torch.from_numpy(mask).cuda()
    out = torch.empty(mask.shape, dtype=torch.int32, device=x.device)
    binding.prof_enable(64)
    try:
        binding.tm_cdt_ws(x, 2, code, out, None)
        torch.cuda.synchronize()
        names = [n for n, _ in binding.prof_read()]
    finally:
        binding.prof_enable(0)
    assert names == ["scan_word.o16", "cdt_l1_scan_final.i16"], names
    full_size_checks(mask, out.cpu().numpy(), "taxicab", 7)


# (batch, spatial, kernel of the last pass): whole taxicab lines of 300, 1000,
# 2000 and 2304 rows (16 or 36 rows per lane, ragged last lanes, 8-line
# groups of 64-, 24-, 8- and 16-wide rows), a 3-D case after the paired tile,
# and 2400 rows (past 36 rows per lane: the whole-line search)
L1_SCAN = [(2, (300, 64), "cdt_l1_scan_final"),
           (1, (1000, 24), "cdt_l1_scan_final"),
           (3, (2000, 8), "cdt_l1_scan_final"),
           (2, (2304, 16), "cdt_l1_scan_final"),
           (2, (300, 20, 16), "cdt_l1_scan_final"),
           (2, (2400, 16), "cdt_line_final")]


@pytest.mark.parametrize("batch,spatial,last", L1_SCAN,
                         ids=["b%d-%s" % (b, "x".join(map(str, s))) for b, s, _ in L1_SCAN])
def test_taxicab_scan_shapes(batch, spatial, last):
    from paper_2608_24738_amd import binding
    mask = rand_mask((batch, 1) + spatial, 0.003, 5000 + sum(spatial))
    mask[(0, 0) + tuple(n // 2 for n in spatial)] = 0
    if batch > 1:
        mask[1] = 1                                # a sample without background
    binding.prof_enable(64)
    try:
        check(mask, len(spatial), "taxicab", "l1 scan")
        names = [n for n, _ in binding.prof_read()]
    finally:
        binding.prof_enable(0)
    assert last in names, names
