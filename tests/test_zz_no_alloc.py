"""GPU test of tm_edt_noalloc, the allocation-free twin of tm_edt_ws: its
workspace is the library's static per-device array.  Called through the
C-ABI, its distances must equal tm_edt_ws's bit for bit (and the oracle's) on
two calls in a row, the second with a smaller input, and the calls must not
change the device memory torch has allocated."""
import ctypes

import numpy as np
import pytest

from gpu_util import announce, check_against_oracle
from oracle import edt_oracle
from paper_2608_24738_amd import workloads

pytestmark = pytest.mark.gpu


def call_noalloc(lib, x, out, stream):
    sh = (ctypes.c_int64 * 2)(*x.shape[1:])
    return lib.tm_edt_noalloc(ctypes.c_void_p(x.data_ptr()), 2, sh, x.shape[0], None,
                              ctypes.c_void_p(out.data_ptr()), None, ctypes.c_void_p(stream))


def test_noalloc_matches_workspace_entry():
    import torch
    from paper_2608_24738_amd import binding
    lib = binding.load()
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream().cuda_stream
    cases = [((512, 512), 32), ((128, 512), 32)]          # the second call smaller
    outs = []
    for spatial, batch in cases:
        mask = workloads.make_mask(2, spatial, batch)[:, 0].copy()
        mask[1] = 1                                         # a sample without background
        x = torch.from_numpy(mask).to(dev)
        announce("tm_edt_noalloc shape=%s" % (mask.shape,))
        out = torch.empty(mask.shape, dtype=torch.float32, device=dev)
        torch.cuda.synchronize()
        before = torch.cuda.memory_allocated(dev)
        binding.prof_enable(64)
        try:
            rc = call_noalloc(lib, x, out, stream)
            torch.cuda.synchronize()
            names = [n for n, _ in binding.prof_read()]
        finally:
            binding.prof_enable(0)
        assert rc == 0, binding.tm_strerror(rc)
        assert torch.cuda.memory_allocated(dev) == before
        assert names == ["scan_word.cost.o16", "order", "line_pair_final.i16"], names
        # the entry point with a caller workspace, on the same input
        need = binding.tm_edt_workspace_size(2, spatial, batch)
        ws = torch.zeros(need // 4, dtype=torch.int32, device=dev)
        ref = torch.empty_like(out)
        binding.tm_edt_ws(x, 2, None, ref, None, ws)
        torch.cuda.synchronize()
        got = out.cpu().numpy()
        assert np.array_equal(got, ref.cpu().numpy()), "tm_edt_noalloc and tm_edt_ws differ"
        ora = edt_oracle.edt(mask, 2, None, want_sq=False, want_dist=True, nthreads=16)
        check_against_oracle(mask, 2, None, {"dist": got}, ora)
        outs.append(got)
    assert len(outs) == 2


def test_noalloc_whole_line_search_order():
    """The order of the whole-line search (units of four 8-column workgroups)
    in the static workspace: 8 x 1024^2 discs, then a smaller 4 x 768 x 2048
    input, each equal to tm_edt_ws's result."""
    import torch
    from paper_2608_24738_amd import binding
    lib = binding.load()
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream().cuda_stream
    for spatial, batch in [((1024, 1024), 8), ((768, 2048), 4)]:
        mask = workloads.make_mask(9, spatial, batch)[:, 0].copy()
        x = torch.from_numpy(mask).to(dev)
        announce("tm_edt_noalloc whole-line search shape=%s" % (mask.shape,))
        out = torch.empty(mask.shape, dtype=torch.float32, device=dev)
        binding.prof_enable(64)
        try:
            rc = call_noalloc(lib, x, out, stream)
            torch.cuda.synchronize()
            names = [n for n, _ in binding.prof_read()]
        finally:
            binding.prof_enable(0)
        assert rc == 0, binding.tm_strerror(rc)
        need = binding.tm_edt_workspace_size(2, spatial, batch)
        assert need > 0
        assert names == ["scan_word.cost.o16", "order", "line_search_final.i16"], names
        ws = torch.zeros(max(1, need // 4), dtype=torch.int32, device=dev)
        ref = torch.empty_like(out)
        binding.tm_edt_ws(x, 2, None, ref, None, ws)
        torch.cuda.synchronize()
        assert np.array_equal(out.cpu().numpy(), ref.cpu().numpy())
