"""Runtime behaviour of the boundary (paper, Section 2.4 "Runtime tests"; the
API surface of Section 2.2.1).

- Work goes on the caller's stream: a transform enqueued on a side stream
  behind a slow producer of its mask sees the produced mask, and a consumer
  enqueued after it on that stream sees the finished result.
- The transforms allocate no device memory.
- The scipy-style wrapper takes any element type (nonzero and NaN are
  foreground) and any strides, with C > 1, and fills pre-allocated outputs
  of any layout.
- tm_mask_nonzero itself: every dtype code, strided views, the bit-pattern
  rule for +0 / -0 / NaN / infinities / subnormals.
Every result is compared with the oracle element by element.
"""
import ctypes

import numpy as np
import pytest

from gpu_util import announce, check_against_oracle
from oracle import edt_oracle
from paper_2608_24738_amd import binding, workloads

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
DEV = "cuda:0"


def oracle(mask, ndim, sampling=None):
    return edt_oracle.edt(mask, ndim, sampling, nthreads=16)


def _slow_work(stream):
    """Keep `stream` busy for a few milliseconds with ordinary kernels."""
    a = torch.randn(2048, 2048, device=DEV)
    with torch.cuda.stream(stream):
        for _ in range(24):
            a = torch.tanh(a @ a * 1e-3)
    return a


def test_side_stream_orders_producer_transform_consumer():
    mask = workloads.make_mask(3, (48, 40, 64), 2)
    want = oracle(mask, 3)
    announce("side stream: producer -> tm_edt / tm_edt_sq -> consumer, shape %s" % (mask.shape,))
    src = torch.from_numpy(mask).to(DEV)
    dst = torch.ones_like(src)                    # all foreground until the producer runs
    dist = torch.empty(mask.shape, dtype=torch.float32, device=DEV)
    sq = torch.empty(mask.shape, dtype=torch.int32, device=DEV)
    torch.cuda.synchronize()
    side = torch.cuda.Stream(device=DEV)          # default priority
    keep = _slow_work(side)
    with torch.cuda.stream(side):
        dst.copy_(src)                            # the producer, behind the slow work
        binding.tm_edt(dst, 3, None, dist, None)  # current stream = side
        binding.tm_edt_sq(dst, 3, sq, None, stream=side)
        doubled = dist * 2.0                      # the consumer
        sq_plus = sq + 1
    side.synchronize()
    del keep
    assert np.array_equal(dist.cpu().numpy(), want["dist"])
    assert np.array_equal(sq.cpu().numpy(), want["sq"])
    assert np.array_equal(doubled.cpu().numpy(), want["dist"] * np.float32(2.0))
    assert np.array_equal(sq_plus.cpu().numpy(), want["sq"] + 1)


def test_wrapper_on_side_stream_with_indices():
    mask = workloads.make_mask(1, (40, 52), 3)
    want = oracle(mask, 2)
    announce("side stream wrapper: distance_transform_edt with indices, shape %s" % (mask.shape,))
    src = torch.from_numpy(mask).to(DEV)
    dst = torch.ones_like(src)
    torch.cuda.synchronize()
    side = torch.cuda.Stream(device=DEV)
    keep = _slow_work(side)
    with torch.cuda.stream(side):
        dst.copy_(src)
        dist, idx = binding.distance_transform_edt(dst, return_indices=True)
    side.synchronize()
    del keep
    res = {"dist": dist.cpu().numpy(), "idx": idx.cpu().numpy(), "sq": None}
    check_against_oracle(mask, 2, None, res, want)


def test_transforms_allocate_nothing():
    mask = workloads.make_mask(3, (64, 64, 64), 2)
    x = torch.from_numpy(mask).to(DEV)
    dist = torch.empty(mask.shape, dtype=torch.float32, device=DEV)
    sq = torch.empty(mask.shape, dtype=torch.int32, device=DEV)
    idx = torch.empty((2, 1, 3, 64, 64, 64), dtype=torch.int32, device=DEV)
    sgn = torch.empty(mask.shape, dtype=torch.float32, device=DEV)
    cdt = torch.empty(mask.shape, dtype=torch.int32, device=DEV)

    def calls():
        binding.tm_edt(x, 3, None, dist, None)
        binding.tm_edt(x, 3, [2.0, 1.0, 0.5], dist, idx)
        binding.tm_edt_sq(x, 3, sq, idx)
        binding.tm_edt_signed(x, 3, sgn)
        binding.tm_cdt(x, 3, 1, cdt)

    announce("no allocation: tm_edt / tm_edt_sq / tm_edt_signed / tm_cdt on (2,1,64,64,64)")
    calls()                                       # first launches load the code objects
    torch.cuda.synchronize()
    alloc0 = torch.cuda.memory_allocated()
    torch.cuda.reset_peak_memory_stats()
    free0, _ = torch.cuda.mem_get_info()
    for _ in range(3):
        calls()
    torch.cuda.synchronize()
    free1, _ = torch.cuda.mem_get_info()
    assert torch.cuda.memory_allocated() == alloc0
    assert torch.cuda.max_memory_allocated() == alloc0
    assert free1 == free0, "device memory in use changed by %d bytes" % (free0 - free1)
    want = oracle(mask, 3)
    assert np.array_equal(sq.cpu().numpy(), want["sq"])


def _noncontig(mask):
    """A non-contiguous (B, C, *S) view whose values equal `mask`."""
    return torch.from_numpy(np.ascontiguousarray(np.swapaxes(mask, -1, -2))).to(DEV).transpose(-1, -2)


def test_wrapper_noncontiguous_input_with_channels():
    rng = np.random.default_rng([7, 1])
    mask = (rng.random((2, 3, 37, 50)) < 0.93).astype(np.uint8)
    mask[1, 2] = 1                                # one sample with no background
    want = oracle(mask, 2)
    x = _noncontig(mask)
    assert not x.is_contiguous()
    announce("wrapper: transposed uint8 input (2,3,37,50), distances + indices")
    dist, idx = binding.distance_transform_edt(x, return_indices=True)
    torch.cuda.synchronize()
    res = {"dist": dist.cpu().numpy(), "idx": idx.cpu().numpy(), "sq": None}
    check_against_oracle(mask, 2, None, res, want)
    sq = binding.distance_transform_edt_sq(x)
    assert np.array_equal(sq.cpu().numpy(), want["sq"])


def test_wrapper_preallocated_outputs():
    rng = np.random.default_rng([7, 2])
    mask = (rng.random((1, 2, 30, 41, 9)) < 0.9).astype(np.uint8)
    samp = (1.5, 1.0, 0.7)
    want = oracle(mask, 3, samp)
    x = torch.from_numpy(mask).to(DEV)
    announce("wrapper: pre-allocated contiguous distances / indices, sampled (1,2,30,41,9)")
    d = torch.full(mask.shape, -7.0, dtype=torch.float32, device=DEV)
    i = torch.full((1, 2, 3, 30, 41, 9), -7, dtype=torch.int32, device=DEV)
    assert binding.distance_transform_edt(x, sampling=samp, return_indices=True, distances=d, indices=i) is None
    torch.cuda.synchronize()
    res = {"dist": d.cpu().numpy(), "idx": i.cpu().numpy(), "sq": None}
    check_against_oracle(mask, 3, samp, res, want)

    announce("wrapper: pre-allocated non-contiguous distances / indices, unit (1,2,30,41,9)")
    want = oracle(mask, 3)
    dbuf = torch.full((1, 2, 9, 41, 30), -7.0, dtype=torch.float32, device=DEV)
    ibuf = torch.full((1, 2, 3, 9, 41, 30), -7, dtype=torch.int32, device=DEV)
    d = dbuf.permute(0, 1, 4, 3, 2)
    i = ibuf.permute(0, 1, 2, 5, 4, 3)
    assert not d.is_contiguous() and not i.is_contiguous()
    assert binding.distance_transform_edt(x, return_indices=True, distances=d, indices=i) is None
    torch.cuda.synchronize()
    res = {"dist": d.cpu().numpy(), "idx": i.cpu().numpy(), "sq": None}
    check_against_oracle(mask, 3, None, res, want)

    announce("wrapper: pre-allocated indices only")
    i2 = torch.empty((1, 2, 3, 30, 41, 9), dtype=torch.int32, device=DEV)
    assert binding.distance_transform_edt(x, return_distances=False, return_indices=True, indices=i2) is None
    torch.cuda.synchronize()
    assert np.array_equal(i2.cpu().numpy(), want["idx"])

    announce("wrapper: pre-allocated chamfer / signed outputs (non-contiguous)")
    cbuf = torch.empty((1, 2, 9, 41, 30), dtype=torch.int32, device=DEV)
    c = cbuf.permute(0, 1, 4, 3, 2)
    assert binding.distance_transform_cdt(x, metric="taxicab", distances=c) is None
    sbuf = torch.empty((1, 2, 9, 41, 30), dtype=torch.float32, device=DEV)
    sg = sbuf.permute(0, 1, 4, 3, 2)
    assert binding.signed_distance_transform(x, distances=sg) is None
    torch.cuda.synchronize()
    assert np.array_equal(c.cpu().numpy(), edt_oracle.cdt(mask, 3, "taxicab"))
    assert np.array_equal(sg.cpu().numpy(), edt_oracle.signed_edt(mask, 3))

    with pytest.raises(RuntimeError):
        binding.distance_transform_edt(x, distances=torch.empty(mask.shape, dtype=torch.float64, device=DEV))
    with pytest.raises(RuntimeError):
        binding.distance_transform_edt(x, return_indices=True,
                                       indices=torch.empty((1, 2, 3, 30, 41, 8), dtype=torch.int32, device=DEV))


def _values(dtype, shape, rng):
    """Random values of `dtype` with many exact zeros (and, for floats, -0.0,
    NaN, infinities and subnormals), plus the foreground mask they define."""
    pick = rng.random(shape)
    if dtype.is_floating_point:
        v = rng.normal(size=shape) * 100.0
        v[pick < 0.05] = 0.0
        v[(pick >= 0.05) & (pick < 0.08)] = -0.0
        v[(pick >= 0.08) & (pick < 0.09)] = np.nan
        v[(pick >= 0.09) & (pick < 0.095)] = np.inf
        v[(pick >= 0.095) & (pick < 0.1)] = -np.inf
        t = torch.from_numpy(v).to(dtype)
        tiny = {torch.float16: 2.0 ** -24, torch.bfloat16: 2.0 ** -133, torch.float32: 2.0 ** -149,
                torch.float64: 2.0 ** -1074}.get(dtype)
        if tiny is not None:
            sub = torch.from_numpy(pick >= 0.995)
            t[sub] = torch.tensor(tiny, dtype=torch.float64).to(dtype)
            t[torch.from_numpy((pick >= 0.99) & (pick < 0.995))] = -torch.tensor(tiny, dtype=torch.float64).to(dtype)
        # the reference predicate on the very values the GPU reads: != 0 (NaN != 0)
        ref = (t.to(torch.float64) != 0).numpy()
    else:
        v = rng.integers(-3, 4, size=shape) if dtype != torch.uint8 and dtype != torch.bool else \
            rng.integers(0, 4, size=shape)
        v[pick < 0.1] = 0
        t = torch.from_numpy(v).to(dtype)
        ref = (t.to(torch.int64) != 0).numpy()
    return t, ref.astype(np.uint8)


DTYPES = ["uint8", "int8", "bool", "int16", "int32", "int64", "float16", "bfloat16", "float32",
          "float64", "float8_e4m3fn", "float8_e5m2", "float8_e4m3fnuz", "float8_e5m2fnuz", "uint16",
          "uint32", "uint64"]


@pytest.mark.parametrize("name", DTYPES)
def test_wrapper_any_dtype(name):
    if not hasattr(torch, name):
        pytest.skip("torch has no %s" % name)
    dtype = getattr(torch, name)
    rng = np.random.default_rng([7, 3, DTYPES.index(name)])
    shape = (2, 2, 23, 65)
    if name.startswith("float8"):
        v = rng.normal(size=shape) * 4.0
        v[rng.random(shape) < 0.1] = 0.0
        v[rng.random(shape) < 0.05] = -0.0
        t = torch.from_numpy(v).to(torch.float32).to(dtype)
        ref = (t.to(torch.float32) != 0).numpy().astype(np.uint8)
    elif name.startswith("uint") and name != "uint8":
        v = rng.integers(0, 5, size=shape)
        v[rng.random(shape) < 0.1] = 0
        t = torch.from_numpy(v.astype(np.int64)).to(dtype)
        ref = (v != 0).astype(np.uint8)
    else:
        t, ref = _values(dtype, shape, rng)
    want = oracle(ref, 2)
    announce("wrapper: %s input %s (contiguous and transposed)" % (name, shape))
    x = t.to(DEV)
    dist, idx = binding.distance_transform_edt(x, return_indices=True)
    torch.cuda.synchronize()
    check_against_oracle(ref, 2, None, {"dist": dist.cpu().numpy(), "idx": idx.cpu().numpy(), "sq": None}, want)
    xt = t.transpose(-1, -2).contiguous().to(DEV).transpose(-1, -2)
    assert not xt.is_contiguous()
    dist2 = binding.distance_transform_edt(xt)
    torch.cuda.synchronize()
    assert np.array_equal(dist2.cpu().numpy(), want["dist"])


def test_mask_predicate_strided_views():
    """tm_mask_nonzero through the C-ABI on strided views: slices with steps,
    broadcast (stride 0) axes, a permuted view, against numpy's x != 0."""
    lib = binding.load()
    rng = np.random.default_rng([7, 4])
    base = rng.normal(size=(6, 40, 70)).astype(np.float32)
    base[rng.random(base.shape) < 0.2] = 0.0
    base[rng.random(base.shape) < 0.05] = -0.0
    base[rng.random(base.shape) < 0.02] = np.nan
    g = torch.from_numpy(base).to(DEV)
    views = {
        "step-slices": (g[1::2, ::3, 5:61:2], base[1::2, ::3, 5:61:2]),
        "permuted": (g.permute(2, 0, 1), base.transpose(2, 0, 1)),
        "broadcast": (g[2:3, 7].expand(5, 70), np.broadcast_to(base[2:3, 7], (5, 70))),
        "one-element": (g[3, 4, 5:6], base[3, 4, 5:6]),
    }
    for name, (v, ref_vals) in views.items():
        announce("tm_mask_nonzero: %s view %s strides %s" % (name, tuple(v.shape), v.stride()))
        out = torch.full((v.numel(),), 7, dtype=torch.uint8, device=DEV)
        binding.tm_mask_nonzero(v, out)
        torch.cuda.synchronize()
        want = (np.asarray(ref_vals) != 0).astype(np.uint8).ravel()
        assert np.array_equal(out.cpu().numpy(), want), name
    # odd output address: byte stores at the ends
    v = g[0, :3, :7]
    out = torch.full((64,), 7, dtype=torch.uint8, device=DEV)
    binding.tm_mask_nonzero(v, out[1:22])
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    assert got[0] == 7 and (got[22:] == 7).all()
    assert np.array_equal(got[1:22], (base[0, :3, :7] != 0).astype(np.uint8).ravel())
    # the output must not overlap the input
    sh = (ctypes.c_int64 * 1)(8)
    assert lib.tm_mask_nonzero(ctypes.c_void_p(g.data_ptr()), 6, 1, sh, None,
                               ctypes.c_void_p(g.data_ptr() + 4), None) == -8
