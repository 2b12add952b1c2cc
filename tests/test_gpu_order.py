"""GPU parity of tm_edt_ws, whose workspace carries a dispatch order for the
column pass of 2-D distance requests with at least 1024 groups of columns:
the row scan estimates each group's work (k_scan_word with the cost
estimate), k_order sorts the groups heaviest first, and the column pass
(k_line_pair16, 16 columns per workgroup, or k_line_search, 8) takes them in
that order.  The
order decides only when each group runs, so every result must equal the
oracle's bit for bit, and equal tm_edt's (no workspace), whatever the
workspace held before the call.  Each case checks which kernels ran.
"""
import numpy as np
import pytest

from gpu_util import announce, check_against_oracle
from oracle import edt_oracle
from paper_2608_24738_amd import workloads

pytestmark = pytest.mark.gpu


def run_ws(mask, ws_fill=None, ws_bytes=None):
    """tm_edt_ws on (batch, n0, n1) ``mask`` with a fresh workspace (zeros,
    or ``ws_fill`` 32-bit words); returns (dist, kernel names, workspace)."""
    import torch
    from paper_2608_24738_amd import binding
    dev = torch.device("cuda:0")
    x = torch.from_numpy(np.ascontiguousarray(mask)).to(dev)
    need = binding.tm_edt_workspace_size(2, mask.shape[1:], mask.shape[0])
    nb = need if ws_bytes is None else ws_bytes
    ws = None
    if nb:
        words = (nb + 3) // 4
        if ws_fill is None:
            ws = torch.zeros(words, dtype=torch.int32, device=dev)
        else:
            ws = torch.from_numpy(np.ascontiguousarray(ws_fill[:words]).view(np.int32)).to(dev)
    d = torch.empty(mask.shape, dtype=torch.float32, device=dev)
    binding.prof_enable(64)
    try:
        binding.tm_edt_ws(x, 2, None, d, None, ws)
        torch.cuda.synchronize()
        names = [n for n, _ in binding.prof_read()]
    finally:
        binding.prof_enable(0)
    return d.cpu().numpy(), names, (None if ws is None else ws.cpu().numpy()), need


def run_plain(mask):
    import torch
    from paper_2608_24738_amd import binding
    dev = torch.device("cuda:0")
    x = torch.from_numpy(np.ascontiguousarray(mask)).to(dev)
    d = torch.empty(mask.shape, dtype=torch.float32, device=dev)
    binding.tm_edt(x, 2, None, d, None)
    torch.cuda.synchronize()
    return d.cpu().numpy()


def check_ordered(mask, tag, ws_fill=None, final="line_pair_final.i16"):
    announce("ordered column pass %s shape=%s" % (tag, mask.shape))
    dist, names, ws, need = run_ws(mask, ws_fill)
    assert need > 0, "this request should take a workspace"
    scan = "scan_word.cost.o16" if final.endswith(".i16") else "scan_word.cost"
    assert names == [scan, "order", final], names
    ora = edt_oracle.edt(mask, 2, None, want_sq=False, want_dist=True, nthreads=16)
    check_against_oracle(mask, 2, None, {"dist": dist}, ora)
    assert np.array_equal(dist, run_plain(mask)), "tm_edt_ws and tm_edt differ"
    groups = need // 8
    order = ws[groups:2 * groups]
    assert np.array_equal(np.sort(order), np.arange(groups)), "order is not a permutation"
    assert not ws[:groups].any(), "counters not cleared"
    return order


def test_full_workload_2():
    mask = workloads.make_mask(2)[:, 0]             # 32 x 512^2 discs
    order = check_ordered(mask, "32x512^2 discs")
    # the first groups dispatched cross more foreground than the last ones
    g = mask.reshape(32, 512, 32, 16).sum(axis=(1, 3)).reshape(-1)
    assert g[order[:64]].mean() > g[order[-64:]].mean()


@pytest.mark.parametrize("p_bg", [0.3, 0.01, 0.0005])
def test_densities(p_bg):
    rng = np.random.default_rng([41, int(p_bg * 1e4)])
    mask = (rng.random((32, 256, 512)) >= p_bg).astype(np.uint8)
    check_ordered(mask, "p_bg=%g" % p_bg)


def test_short_batch_32_position_words():
    # 32 x 128 x 512: few enough rows that the scan takes 32-position words
    mask = workloads.make_mask(2, (128, 512), 32)[:, 0]
    check_ordered(mask, "32x128x512")


def test_whole_line_search_full_workload_9():
    # 8 x 1024^2 discs: columns of 1024 rows, 8 per workgroup of k_line_search
    mask = workloads.make_mask(9)[:, 0]
    check_ordered(mask, "8x1024^2 discs", final="line_search_final.i16")


@pytest.mark.parametrize("p_bg", [0.01, 0.0002])
def test_whole_line_search_densities(p_bg):
    rng = np.random.default_rng([45, int(p_bg * 1e4)])
    mask = (rng.random((8, 1024, 1024)) >= p_bg).astype(np.uint8)
    mask[3] = 1                      # no background: the virtual element
    check_ordered(mask, "1024^2 p_bg=%g" % p_bg, final="line_search_final.i16")


def test_samples_without_background_and_ties():
    rng = np.random.default_rng(43)
    mask = (rng.random((32, 256, 512)) >= 0.002).astype(np.uint8)
    mask[0] = 1                      # no background: the virtual element
    mask[5] = 0                      # all background
    mask[9] = 1
    mask[9, :, 100] = 0              # one background column: equal costs along it
    check_ordered(mask, "empty samples")


def test_workspace_contents_do_not_matter():
    mask = workloads.make_mask(2, (256, 512), 32)[:, 0]
    rng = np.random.default_rng(44)
    junk = rng.integers(0, 2 ** 32, size=2 * 1024, dtype=np.uint64).astype(np.uint32)
    check_ordered(mask, "junk workspace", ws_fill=junk)
    ones = np.full(2 * 1024, 0xffffffff, np.uint32)   # counters that wrap when added to
    check_ordered(mask, "all-ones workspace", ws_fill=ones)


def test_small_or_missing_workspace_runs_unordered():
    mask = workloads.make_mask(2, (256, 512), 32)[:, 0]
    announce("workspace too small shape=%s" % (mask.shape,))
    want = run_plain(mask)
    for nb in (0, 8):
        dist, names, _, need = run_ws(mask, ws_bytes=nb)
        assert names == ["scan_word.o16", "line_pair_final.i16"], names
        assert np.array_equal(dist, want)


def test_reuse_across_calls_and_shapes():
    # one workspace, masks of different sizes in turn: each call orders its own groups
    import torch
    from paper_2608_24738_amd import binding
    dev = torch.device("cuda:0")
    ws = torch.zeros(2 * 1024, dtype=torch.int32, device=dev)
    for k, (batch, n0) in enumerate([(32, 512), (32, 128), (32, 256), (32, 512)]):
        mask = workloads.make_mask(2, (n0, 512), batch)[:, 0].copy()
        mask[k % batch] = 1
        announce("reuse %d shape=%s" % (k, mask.shape))
        x = torch.from_numpy(mask).to(dev)
        d = torch.empty(mask.shape, dtype=torch.float32, device=dev)
        binding.tm_edt_ws(x, 2, None, d, None, ws)
        torch.cuda.synchronize()
        ora = edt_oracle.edt(mask, 2, None, want_sq=False, want_dist=True, nthreads=16)
        check_against_oracle(mask, 2, None, {"dist": d.cpu().numpy()}, ora)
        groups = batch * 512 // 16
        assert not ws[:groups].cpu().numpy().any()


def test_scipy_wrapper_uses_the_workspace():
    import torch
    from paper_2608_24738_amd import binding
    mask = workloads.make_mask(2, (256, 512), 32)
    announce("wrapper shape=%s" % (mask.shape,))
    x = torch.from_numpy(mask).cuda()
    binding.prof_enable(64)
    try:
        d = binding.distance_transform_edt(x)
        torch.cuda.synchronize()
        names = [n for n, _ in binding.prof_read()]
    finally:
        binding.prof_enable(0)
    assert "order" in names, names
    ora = edt_oracle.edt(mask[:, 0], 2, None, want_sq=False, want_dist=True, nthreads=16)
    assert np.array_equal(d.cpu().numpy()[:, 0], ora["dist"])


def test_misaligned_buffers_run_unordered():
    # the row scan that estimates the costs needs 16-byte aligned input and
    # output; a misaligned input runs the other scans, without an order
    import torch
    from paper_2608_24738_amd import binding
    dev = torch.device("cuda:0")
    mask = workloads.make_mask(2, (256, 512), 32)[:, 0].copy()
    announce("misaligned input shape=%s" % (mask.shape,))
    big = torch.empty(mask.size + 16, dtype=torch.uint8, device=dev)
    x = big[1:1 + mask.size].view(mask.shape)
    x.copy_(torch.from_numpy(mask).to(dev))
    assert x.data_ptr() % 16 == 1
    need = binding.tm_edt_workspace_size(2, mask.shape[1:], mask.shape[0])
    assert need > 0
    ws = torch.zeros(need // 4, dtype=torch.int32, device=dev)
    d = torch.empty(mask.shape, dtype=torch.float32, device=dev)
    binding.prof_enable(64)
    try:
        binding.tm_edt_ws(x, 2, None, d, None, ws)
        torch.cuda.synchronize()
        names = [n for n, _ in binding.prof_read()]
    finally:
        binding.prof_enable(0)
    assert "order" not in names and not any(n.startswith("scan_word.cost") for n in names), names
    ora = edt_oracle.edt(mask, 2, None, want_sq=False, want_dist=True, nthreads=16)
    check_against_oracle(mask, 2, None, {"dist": d.cpu().numpy()}, ora)
    assert not ws.cpu().numpy().any()
