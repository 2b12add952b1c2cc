"""The C-ABI library: exported symbols, host-side checks and argument
validation.  Every call here is rejected on the host before any HIP call, so
these run without a GPU."""
import ctypes
import glob
import os
import re

import pytest

from paper_2608_24738_amd import binding, build as hip_build

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

TM_OK, TM_ERR_NDIM, TM_ERR_SHAPE, TM_ERR_BATCH, TM_ERR_NULL = 0, -1, -2, -3, -4
TM_ERR_NO_OUTPUT, TM_ERR_SAMPLING, TM_ERR_TOO_LARGE, TM_ERR_ALIAS = -5, -6, -7, -8
TM_ERR_UNSUPPORTED, TM_ERR_HIP, TM_ERR_METRIC, TM_ERR_DTYPE = -9, -10, -11, -12
TM_ERR_WORKSPACE = -13

FAKE_IN = 0x100000           # never dereferenced: every call below fails validation
FAKE_OUT = 0x40000000
FAKE_IDX = 0x80000000


@pytest.fixture(scope="module")
def lib():
    if hip_build.is_stale():
        hip_build.build()
    return binding.load()


def declared_functions():
    names = []
    for h in glob.glob(os.path.join(ROOT, "include", "*.h")):
        text = open(h).read()
        names += re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(tm_\w+)\s*\(", text, re.M)
    return sorted(set(names))


def test_every_declared_symbol_is_exported(lib):
    names = declared_functions()
    assert {"tm_edt", "tm_edt_sq", "tm_edt_signed", "tm_dt_bf", "tm_cdt", "tm_mask_nonzero",
            "tm_strerror"} <= set(names)
    for n in names:
        assert hasattr(lib, n), n


def test_host_division_constants(lib):
    assert lib.tm_selftest_host() == 0


def test_strerror_covers_every_status(lib):
    for s in range(0, -14, -1):
        msg = binding.tm_strerror(s)
        assert msg and msg != "unknown status", s
    assert binding.tm_strerror(-99) == "unknown status"


def call_edt(lib, shape, batch=1, sampling=None, inp=FAKE_IN, dist=FAKE_OUT, idx=None, ndim=None):
    nd = len(shape) if ndim is None else ndim
    sh = (ctypes.c_int64 * max(len(shape), 1))(*shape) if shape is not None else None
    samp = (ctypes.c_double * len(sampling))(*sampling) if sampling is not None else None
    return lib.tm_edt(inp and ctypes.c_void_p(inp), nd, sh, batch, samp,
                      dist and ctypes.c_void_p(dist), idx and ctypes.c_void_p(idx), None)


def call_sq(lib, shape, batch=1, inp=FAKE_IN, sq=FAKE_OUT, idx=None):
    sh = (ctypes.c_int64 * len(shape))(*shape)
    return lib.tm_edt_sq(ctypes.c_void_p(inp), len(shape), sh, batch,
                         sq and ctypes.c_void_p(sq), idx and ctypes.c_void_p(idx), None)


def test_rank_limits(lib):
    assert call_edt(lib, [4] * 9) == TM_ERR_NDIM
    assert call_edt(lib, [4], ndim=0) == TM_ERR_NDIM


def test_shape_and_batch(lib):
    assert call_edt(lib, None, ndim=2) == TM_ERR_SHAPE
    assert call_edt(lib, [4, 0]) == TM_ERR_SHAPE
    assert call_edt(lib, [4, -3]) == TM_ERR_SHAPE
    assert call_edt(lib, [4, 4], batch=0) == TM_ERR_BATCH


def test_null_input_and_no_output(lib):
    assert call_edt(lib, [4, 4], inp=0) == TM_ERR_NULL
    assert call_edt(lib, [4, 4], dist=0, idx=0) == TM_ERR_NO_OUTPUT
    assert call_sq(lib, [4, 4], sq=0, idx=0) == TM_ERR_NO_OUTPUT


@pytest.mark.parametrize("bad", [0.0, -1.0, float("inf"), float("nan")])
def test_sampling_must_be_positive_and_finite(lib, bad):
    assert call_edt(lib, [4, 4], sampling=[1.0, bad]) == TM_ERR_SAMPLING


def test_too_large(lib):
    assert call_edt(lib, [1 << 16, 1 << 15]) == TM_ERR_TOO_LARGE          # 2^31 per sample
    assert call_edt(lib, [1 << 10, 1 << 10], batch=1 << 12) == TM_ERR_TOO_LARGE  # 2^32 total
    assert call_sq(lib, [50000, 2]) == TM_ERR_TOO_LARGE                    # sum of n^2 >= 2^31


def test_overlapping_buffers(lib):
    assert call_edt(lib, [16, 16], dist=FAKE_IN + 100) == TM_ERR_ALIAS
    assert call_edt(lib, [16, 16], dist=FAKE_OUT, idx=FAKE_OUT + 4) == TM_ERR_ALIAS
    assert call_sq(lib, [16, 16], sq=FAKE_OUT, idx=FAKE_OUT + 512) == TM_ERR_ALIAS


FAKE_WS = 0x20000000


def call_edt_ws(lib, shape, batch=1, sampling=None, inp=FAKE_IN, dist=FAKE_OUT, idx=None, ws=FAKE_WS,
                ws_bytes=1 << 16):
    sh = (ctypes.c_int64 * len(shape))(*shape)
    samp = (ctypes.c_double * len(shape))(*sampling) if sampling else None
    return lib.tm_edt_ws(ctypes.c_void_p(inp), len(shape), sh, batch, samp, dist and ctypes.c_void_p(dist),
                         idx and ctypes.c_void_p(idx), ws and ctypes.c_void_p(ws), ws_bytes, None)


def test_workspace_entry_checks(lib):
    # tm_edt's checks first, then the workspace's own: 4-byte alignment, and
    # no overlap with the input or outputs (all refused before any HIP call)
    assert call_edt_ws(lib, [512, 512], batch=0) == TM_ERR_BATCH
    assert call_edt_ws(lib, [512, 512], dist=None) == TM_ERR_NO_OUTPUT
    assert call_edt_ws(lib, [512, 512], sampling=[1.0, -1.0]) == TM_ERR_SAMPLING
    assert call_edt_ws(lib, [512, 512], ws=FAKE_WS + 2) == TM_ERR_WORKSPACE
    assert call_edt_ws(lib, [512, 512], ws=FAKE_IN + 4096) == TM_ERR_ALIAS
    assert call_edt_ws(lib, [512, 512], ws=FAKE_OUT + 64, ws_bytes=8) == TM_ERR_ALIAS
    assert call_edt_ws(lib, [512, 512], ws=FAKE_OUT - 8, ws_bytes=16) == TM_ERR_ALIAS


def test_workspace_size(lib):
    # 8 bytes per group of columns (16 per workgroup of the packed pass, 32
    # for four workgroups of 8 of the whole-line search) for 2-D distance
    # requests with at least 1024 workgroups; nothing for other requests
    size = binding.tm_edt_workspace_size
    assert size(2, (512, 512), 32) == 8 * 32 * 512 // 16
    assert size(2, (512, 512), 32, (1.0, 1.0)) == 8 * 1024          # unit sampling spelled out
    assert size(2, (128, 512), 32) == 8 * 32 * 512 // 16            # 32-position row words
    assert size(2, (1024, 1024), 8) == 8 * 8 * 1024 // 32           # whole-line search: units of 4 x 8 lines
    assert size(2, (512, 512), 512) == 8 * 16384                     # the most groups one order holds
    assert size(2, (512, 512), 16) == 0                              # 512 groups: no order
    assert size(2, (512, 512), 32, None, True) == 0                  # indices: other passes
    assert size(2, (512, 512), 32, (1.0, 2.0)) == 0                  # sampled
    assert size(3, (128, 128, 128), 8) == 0                          # 3-D
    assert size(2, (64, 64), 100) == 0                               # one workgroup per sample
    assert size(2, (2048, 2048), 2) == 0                             # rows past 256 groups
    assert size(2, (256, 256), 8) == 0                               # too few groups to order
    assert size(2, (512, 512), 513) == 0                             # more groups than one order holds
    assert size(2, (512, 512), 0) == 0                               # rejected arguments
    assert size(9, (1,) * 9, 1) == 0


def test_chamfer_workspace(lib):
    size = binding.tm_cdt_workspace_size
    assert size(2, (1024, 1024), 8, 2) == 8 * 8 * 1024 // 32        # units of four 8-column workgroups
    assert size(2, (1024, 1024), 8, 1) == 0                          # taxicab: prefix minima, even work
    assert size(2, (256, 256), 8, 2) == 0                            # 256 workgroups: no order
    assert size(3, (64, 64, 64), 8, 2) == 0
    assert size(2, (1024, 1024), 8, 0) == 0                          # not a chamfer metric
    sh = (ctypes.c_int64 * 2)(1024, 1024)
    def call(metric, ws):
        return lib.tm_cdt_ws(ctypes.c_void_p(FAKE_IN), 2, sh, 8, metric, ctypes.c_void_p(FAKE_OUT),
                             ctypes.c_void_p(ws), 4096, None)
    assert call(0, FAKE_WS) == TM_ERR_METRIC
    assert call(2, FAKE_WS + 2) == TM_ERR_WORKSPACE
    assert call(2, FAKE_IN + 64) == TM_ERR_ALIAS


def test_static_workspace_limit(lib):
    # tm_edt_noalloc refuses, on the host, requests whose dispatch order needs
    # more than its 64 KiB static workspace (8192 groups of 16 columns)
    def call(shape, batch):
        sh = (ctypes.c_int64 * len(shape))(*shape)
        return lib.tm_edt_noalloc(ctypes.c_void_p(FAKE_IN), len(shape), sh, batch, None,
                                  ctypes.c_void_p(FAKE_OUT), None, None)
    assert binding.tm_edt_workspace_size(2, (512, 512), 257) == 8 * 8224 > 65536
    assert call([512, 512], 257) == TM_ERR_WORKSPACE
    assert call([512, 512], 0) == TM_ERR_BATCH
    sh = (ctypes.c_int64 * 2)(512, 512)
    assert lib.tm_edt_noalloc(ctypes.c_void_p(FAKE_IN), 2, sh, 1, None, None, None, None) == TM_ERR_NO_OUTPUT


def test_remaining_line_length_limits(lib):
    # The exact transform takes strided lines of any length (the envelope of a
    # line too long for LDS lives in the line's own storage); the limits left
    # are the signed transform's whole-line tile (32-bit, one line per
    # workgroup: about 40 700 elements) and the chessboard chamfer pass past
    # 16-bit values (about 40 700 elements).  These calls are refused on the
    # host; nothing is launched.
    assert call_cdt(lib, [70000, 2], metric=2) == TM_ERR_UNSUPPORTED
    sh = (ctypes.c_int64 * 2)(45000, 3)
    assert lib.tm_edt_signed(ctypes.c_void_p(FAKE_IN), 2, sh, 1, ctypes.c_void_p(FAKE_OUT), None) \
        == TM_ERR_UNSUPPORTED


def test_binding_rejects_bad_python_arguments():
    torch = pytest.importorskip("torch")
    x = torch.zeros((1, 1, 4, 4), dtype=torch.uint8)
    with pytest.raises(ValueError):
        binding.tm_edt(x, 2, out_dist=torch.empty(16))                    # not a GPU tensor
    with pytest.raises(RuntimeError):
        binding.distance_transform_edt(x, return_distances=False, return_indices=False)
    with pytest.raises(RuntimeError):
        binding.distance_transform_edt(x, sampling=[1.0, 2.0, 3.0])
    with pytest.raises(ValueError):
        binding.distance_transform_edt(x.float())                         # any dtype, but on the GPU
    with pytest.raises(TypeError):
        binding._as_mask(torch.zeros((1, 1, 4, 4), dtype=torch.complex64, device="meta"))
    with pytest.raises(ValueError):
        binding.distance_transform_edt(torch.zeros((4, 4), dtype=torch.uint8))


def call_bf(lib, shape, metric=0, batch=1, sampling=None, inp=FAKE_IN, dist=FAKE_OUT, idx=None):
    sh = (ctypes.c_int64 * len(shape))(*shape)
    samp = (ctypes.c_double * len(sampling))(*sampling) if sampling is not None else None
    return lib.tm_dt_bf(ctypes.c_void_p(inp), len(shape), sh, batch, metric, samp,
                        dist and ctypes.c_void_p(dist), idx and ctypes.c_void_p(idx), None)


def test_brute_force_argument_checks(lib):
    assert call_bf(lib, [4, 4], metric=3) == TM_ERR_METRIC
    assert call_bf(lib, [4, 4], metric=-1) == TM_ERR_METRIC
    assert call_bf(lib, [4, 4], dist=0) == TM_ERR_NO_OUTPUT
    assert call_bf(lib, [4, 0]) == TM_ERR_SHAPE
    assert call_bf(lib, [4, 4], sampling=[1.0, 0.0]) == TM_ERR_SAMPLING
    assert call_bf(lib, [16, 16], dist=FAKE_IN + 8) == TM_ERR_ALIAS


def call_cdt(lib, shape, metric=1, batch=1, inp=FAKE_IN, dist=FAKE_OUT):
    sh = (ctypes.c_int64 * len(shape))(*shape)
    return lib.tm_cdt(ctypes.c_void_p(inp), len(shape), sh, batch, metric,
                      dist and ctypes.c_void_p(dist), None)


def test_chamfer_argument_checks(lib):
    assert call_cdt(lib, [4, 4], metric=0) == TM_ERR_METRIC       # no euclidean chamfer
    assert call_cdt(lib, [4, 4], metric=3) == TM_ERR_METRIC
    assert call_cdt(lib, [4, 4], dist=0) == TM_ERR_NO_OUTPUT
    assert call_cdt(lib, [4, 0]) == TM_ERR_SHAPE
    assert call_cdt(lib, [4, 4], batch=0) == TM_ERR_BATCH
    assert call_cdt(lib, [4] * 9) == TM_ERR_NDIM
    assert call_cdt(lib, [16, 16], dist=FAKE_IN + 8) == TM_ERR_ALIAS
    assert call_cdt(lib, [1 << 16, 1 << 15]) == TM_ERR_TOO_LARGE
    # no bound on squared extents (values are sums, not squares); taxicab
    # lines of any length run, chessboard lines past the 16-bit whole-line
    # tile with values beyond 16 bits (about 40 700 elements) are refused
    assert call_cdt(lib, [70000, 2], metric=2) == TM_ERR_UNSUPPORTED
    assert call_cdt(lib, [100000, 3], metric=2) == TM_ERR_UNSUPPORTED


def test_chamfer_binding_checks():
    torch = pytest.importorskip("torch")
    x = torch.zeros((1, 1, 4, 4), dtype=torch.uint8)
    with pytest.raises(ValueError):
        binding.distance_transform_cdt(x, metric="euclidean")
    with pytest.raises(ValueError):
        binding.tm_cdt(x, 2, 1, torch.empty(16, dtype=torch.int32))       # not a GPU tensor
    with pytest.raises(ValueError):
        binding.distance_transform_cdt(x, distances=torch.empty((1, 1, 4, 4)))   # CPU input
    # pre-allocated outputs of the wrong dtype or shape: scipy's RuntimeError
    with pytest.raises(RuntimeError):
        binding._out_buffer(torch.empty((1, 1, 4, 4)), (1, 1, 4, 4), torch.int32, x.device, "distances")
    with pytest.raises(RuntimeError):
        binding._out_buffer(torch.empty((1, 1, 4, 5), dtype=torch.int32), (1, 1, 4, 4), torch.int32,
                            x.device, "distances")


def test_signed_argument_checks(lib):
    def call(shape, batch=1, inp=FAKE_IN, dist=FAKE_OUT, nd=None):
        sh = (ctypes.c_int64 * len(shape))(*shape)
        return lib.tm_edt_signed(inp and ctypes.c_void_p(inp), len(shape) if nd is None else nd, sh, batch,
                                 dist and ctypes.c_void_p(dist), None)
    assert call([4, 4], dist=0) == TM_ERR_NO_OUTPUT
    assert call([4, 4], inp=0) == TM_ERR_NULL
    assert call([4, 4], batch=0) == TM_ERR_BATCH
    assert call([4, 0]) == TM_ERR_SHAPE
    assert call([4] * 9) == TM_ERR_NDIM
    assert call([16, 16], dist=FAKE_IN + 4) == TM_ERR_ALIAS
    assert call([50000, 2]) == TM_ERR_TOO_LARGE          # sum of n^2 >= 2^31
    assert call([45000, 3]) == TM_ERR_UNSUPPORTED        # strided line past the one-line LDS tile


def call_mask(lib, shape, dtype=6, strides=None, inp=FAKE_IN, out=FAKE_OUT, ndim=None):
    nd = len(shape) if ndim is None else ndim
    sh = (ctypes.c_int64 * max(len(shape), 1))(*shape) if shape is not None else None
    st = (ctypes.c_int64 * len(strides))(*strides) if strides is not None else None
    return lib.tm_mask_nonzero(inp and ctypes.c_void_p(inp), dtype, nd, sh, st,
                               out and ctypes.c_void_p(out), None)


def test_mask_predicate_argument_checks(lib):
    assert call_mask(lib, [4, 4], dtype=9) == TM_ERR_DTYPE
    assert call_mask(lib, [4, 4], dtype=-1) == TM_ERR_DTYPE
    assert call_mask(lib, [4] * 17) == TM_ERR_NDIM
    assert call_mask(lib, [4], ndim=0) == TM_ERR_NDIM
    assert call_mask(lib, None, ndim=2) == TM_ERR_SHAPE
    assert call_mask(lib, [4, 0]) == TM_ERR_SHAPE
    assert call_mask(lib, [4, 4], strides=[16, -4]) == TM_ERR_SHAPE
    assert call_mask(lib, [4, 4], inp=0) == TM_ERR_NULL
    assert call_mask(lib, [4, 4], out=0) == TM_ERR_NO_OUTPUT
    assert call_mask(lib, [1 << 16, 1 << 16], dtype=0) == TM_ERR_TOO_LARGE
    # the output may not overlap the bytes the strided view reads
    assert call_mask(lib, [4, 4], dtype=6, out=FAKE_IN + 60) == TM_ERR_ALIAS
    assert call_mask(lib, [4, 4], dtype=6, strides=[64, 4], out=FAKE_IN + 200) == TM_ERR_ALIAS
