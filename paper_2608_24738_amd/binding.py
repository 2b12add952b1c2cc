"""Python binding of ``libtm_edt.so``: argument marshalling only.

Every step of the transform runs in the library's HIP kernels; this module
turns torch tensors into device pointers, shapes and the current HIP stream,
and turns status codes into exceptions.  There is no fallback: if the library
is missing, every call raises.

Entry points with the C names (``tm_edt``, ``tm_edt_ws``, ``tm_edt_noalloc``,
``tm_edt_workspace_size``, ``tm_cdt_ws``, ``tm_cdt_workspace_size``,
``tm_edt_sq``, ``tm_edt_signed``,
``tm_dt_bf``, ``tm_cdt``, ``tm_mask_nonzero``, ``tm_strerror``) plus ``scipy.ndimage``-style
wrappers (``distance_transform_edt``, ``distance_transform_bf``,
``distance_transform_cdt``, ``signed_distance_transform``) over
(B, C, *spatial) tensors (paper, Section 2.2.1).
"""
from __future__ import annotations

import ctypes
import os
import threading

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libtm_edt.so")
_lock = threading.Lock()
_lib = None

TM_OK = 0


class TMError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__("%s failed: %s (status %d)" % (where, tm_strerror(status), status))


def load() -> ctypes.CDLL:
    """Open the library (once). Raises if it has not been built."""
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(LIB_PATH):
                raise RuntimeError(
                    "libtm_edt.so is not built (expected at %s); run "
                    "`python -m paper_2608_24738_amd.build` or __graft_entry__.build()" % LIB_PATH)
            lib = ctypes.CDLL(LIB_PATH)
            vp, i32, i64 = ctypes.c_void_p, ctypes.c_int, ctypes.c_int64
            lib.tm_edt.restype = i32
            lib.tm_edt.argtypes = [vp, i32, vp, i64, vp, vp, vp, vp]
            lib.tm_edt_ws.restype = i32
            lib.tm_edt_ws.argtypes = [vp, i32, vp, i64, vp, vp, vp, vp, ctypes.c_size_t, vp]
            lib.tm_cdt_ws.restype = i32
            lib.tm_cdt_ws.argtypes = [vp, i32, vp, i64, i32, vp, vp, ctypes.c_size_t, vp]
            lib.tm_cdt_workspace_size.restype = ctypes.c_size_t
            lib.tm_cdt_workspace_size.argtypes = [i32, vp, i64, i32]
            lib.tm_edt_noalloc.restype = i32
            lib.tm_edt_noalloc.argtypes = [vp, i32, vp, i64, vp, vp, vp, vp]
            lib.tm_edt_workspace_size.restype = ctypes.c_size_t
            lib.tm_edt_workspace_size.argtypes = [i32, vp, i64, vp, i32]
            lib.tm_edt_sq.restype = i32
            lib.tm_edt_sq.argtypes = [vp, i32, vp, i64, vp, vp, vp]
            lib.tm_dt_bf.restype = i32
            lib.tm_dt_bf.argtypes = [vp, i32, vp, i64, i32, vp, vp, vp, vp]
            lib.tm_edt_signed.restype = i32
            lib.tm_edt_signed.argtypes = [vp, i32, vp, i64, vp, vp]
            lib.tm_cdt.restype = i32
            lib.tm_cdt.argtypes = [vp, i32, vp, i64, i32, vp, vp]
            lib.tm_strerror.restype = ctypes.c_char_p
            lib.tm_strerror.argtypes = [i32]
            lib.tm_prof_enable.restype = i32
            lib.tm_prof_enable.argtypes = [i32]
            lib.tm_prof_count.restype = i32
            lib.tm_prof_count.argtypes = []
            lib.tm_prof_read.restype = i32
            lib.tm_prof_read.argtypes = [i32, ctypes.POINTER(ctypes.c_char_p),
                                         ctypes.POINTER(ctypes.c_float)]
            lib.tm_prof_launch.restype = i32
            lib.tm_prof_launch.argtypes = [i32, ctypes.POINTER(ctypes.c_int64)]
            lib.tm_selftest_host.restype = i32
            lib.tm_selftest_host.argtypes = []
            lib.tm_mask_nonzero.restype = i32
            lib.tm_mask_nonzero.argtypes = [vp, i32, i32, vp, vp, vp, vp]
            _lib = lib
    return _lib


def tm_strerror(status: int) -> str:
    return load().tm_strerror(int(status)).decode()


def _stream_handle(stream) -> int:
    if stream is None:
        stream = torch.cuda.current_stream()
    return int(stream.cuda_stream)


def _shape_args(x: torch.Tensor, ndim: int):
    if x.dim() < ndim:
        raise ValueError("input has fewer than ndim=%d dimensions" % ndim)
    spatial = tuple(int(s) for s in x.shape[x.dim() - ndim:])
    batch = 1
    for s in x.shape[:x.dim() - ndim]:
        batch *= int(s)
    return spatial, batch


def _check_mask(in_u8: torch.Tensor):
    if not in_u8.is_cuda:
        raise ValueError("input must be a ROCm (cuda) tensor")
    if in_u8.dtype not in (torch.uint8, torch.bool):
        raise TypeError("the C entry points read a uint8 or bool mask (nonzero = foreground); got %s; "
                        "the scipy-style wrappers accept any dtype" % in_u8.dtype)
    if not in_u8.is_contiguous():
        raise ValueError("tm_edt needs a contiguous input")


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _check_out(t, dtype, numel, name, dev):
    if t is None:
        return
    if t.dtype != dtype or not t.is_contiguous() or t.numel() != numel or t.device != dev:
        raise ValueError("%s must be a contiguous %s tensor of %d elements on %s"
                         % (name, dtype, numel, dev))


def tm_edt(in_u8: torch.Tensor, ndim: int, sampling=None, out_dist=None, out_idx=None,
           stream=None) -> None:
    """Calls tm_edt on (batch..., *spatial) ``in_u8``; outputs are filled in place."""
    _check_mask(in_u8)
    spatial, batch = _shape_args(in_u8, ndim)
    vox = in_u8.numel() // max(batch, 1)
    _check_out(out_dist, torch.float32, batch * vox, "out_dist", in_u8.device)
    _check_out(out_idx, torch.int32, batch * vox * ndim, "out_idx", in_u8.device)
    shape = (ctypes.c_int64 * ndim)(*spatial)
    samp = None
    if sampling is not None:
        samp = (ctypes.c_double * ndim)(*[float(s) for s in sampling])
    with torch.cuda.device(in_u8.device):
        st = _stream_handle(stream)
        rc = load().tm_edt(_ptr(in_u8), ndim, shape, batch, samp, _ptr(out_dist), _ptr(out_idx),
                           ctypes.c_void_p(st))
    if rc != TM_OK:
        raise TMError(rc, "tm_edt")


def tm_edt_workspace_size(ndim: int, spatial, batch: int, sampling=None, with_indices=False) -> int:
    """Calls tm_edt_workspace_size: bytes of workspace tm_edt_ws uses (0: none)."""
    shape = (ctypes.c_int64 * ndim)(*[int(v) for v in spatial])
    samp = None
    if sampling is not None:
        samp = (ctypes.c_double * ndim)(*[float(v) for v in sampling])
    return int(load().tm_edt_workspace_size(ndim, shape, int(batch), samp, 1 if with_indices else 0))


def tm_edt_ws(in_u8: torch.Tensor, ndim: int, sampling=None, out_dist=None, out_idx=None,
              workspace=None, stream=None) -> None:
    """Calls tm_edt_ws: tm_edt with ``workspace`` (a device tensor, any dtype,
    or None) for the dispatch order of its column pass."""
    _check_mask(in_u8)
    spatial, batch = _shape_args(in_u8, ndim)
    vox = in_u8.numel() // max(batch, 1)
    _check_out(out_dist, torch.float32, batch * vox, "out_dist", in_u8.device)
    _check_out(out_idx, torch.int32, batch * vox * ndim, "out_idx", in_u8.device)
    nbytes = 0
    if workspace is not None:
        if workspace.device != in_u8.device or not workspace.is_contiguous():
            raise ValueError("workspace must be a contiguous tensor on %s" % in_u8.device)
        nbytes = workspace.numel() * workspace.element_size()
    shape = (ctypes.c_int64 * ndim)(*spatial)
    samp = None
    if sampling is not None:
        samp = (ctypes.c_double * ndim)(*[float(v) for v in sampling])
    with torch.cuda.device(in_u8.device):
        st = _stream_handle(stream)
        rc = load().tm_edt_ws(_ptr(in_u8), ndim, shape, batch, samp, _ptr(out_dist), _ptr(out_idx),
                              _ptr(workspace), nbytes, ctypes.c_void_p(st))
    if rc != TM_OK:
        raise TMError(rc, "tm_edt_ws")


def tm_edt_noalloc(in_u8: torch.Tensor, ndim: int, sampling=None, out_dist=None, out_idx=None,
                   stream=None) -> None:
    """Calls tm_edt_noalloc: tm_edt_ws with the library's static workspace."""
    _check_mask(in_u8)
    spatial, batch = _shape_args(in_u8, ndim)
    vox = in_u8.numel() // max(batch, 1)
    _check_out(out_dist, torch.float32, batch * vox, "out_dist", in_u8.device)
    _check_out(out_idx, torch.int32, batch * vox * ndim, "out_idx", in_u8.device)
    shape = (ctypes.c_int64 * ndim)(*spatial)
    samp = None
    if sampling is not None:
        samp = (ctypes.c_double * ndim)(*[float(v) for v in sampling])
    with torch.cuda.device(in_u8.device):
        st = _stream_handle(stream)
        rc = load().tm_edt_noalloc(_ptr(in_u8), ndim, shape, batch, samp, _ptr(out_dist), _ptr(out_idx),
                                   ctypes.c_void_p(st))
    if rc != TM_OK:
        raise TMError(rc, "tm_edt_noalloc")


# Workspaces of the scipy-style wrapper, one per (device, stream): calls on one
# stream run in order, so they can share it.
_workspaces = {}


def _workspace(dev, nbytes: int, stream=None):
    if nbytes <= 0:
        return None
    with torch.cuda.device(dev):
        key = (dev.index, _stream_handle(stream))
    with _lock:
        ws = _workspaces.get(key)
        if ws is None or ws.numel() * 4 < nbytes:
            ws = torch.zeros((nbytes + 3) // 4, dtype=torch.int32, device=dev)
            _workspaces[key] = ws
    return ws


def tm_edt_sq(in_u8: torch.Tensor, ndim: int, out_sq=None, out_idx=None, stream=None) -> None:
    """Calls tm_edt_sq (exact int32 squared distances, unit sampling)."""
    _check_mask(in_u8)
    spatial, batch = _shape_args(in_u8, ndim)
    vox = in_u8.numel() // max(batch, 1)
    _check_out(out_sq, torch.int32, batch * vox, "out_sq", in_u8.device)
    _check_out(out_idx, torch.int32, batch * vox * ndim, "out_idx", in_u8.device)
    shape = (ctypes.c_int64 * ndim)(*spatial)
    with torch.cuda.device(in_u8.device):
        st = _stream_handle(stream)
        rc = load().tm_edt_sq(_ptr(in_u8), ndim, shape, batch, _ptr(out_sq), _ptr(out_idx),
                              ctypes.c_void_p(st))
    if rc != TM_OK:
        raise TMError(rc, "tm_edt_sq")


METRICS = {"euclidean": 0, "taxicab": 1, "chessboard": 2}


def tm_dt_bf(in_u8: torch.Tensor, ndim: int, metric: int, sampling=None, out_dist=None,
             out_idx=None, stream=None) -> None:
    """Calls tm_dt_bf (brute-force transform, metric code 0/1/2)."""
    _check_mask(in_u8)
    spatial, batch = _shape_args(in_u8, ndim)
    vox = in_u8.numel() // max(batch, 1)
    _check_out(out_dist, torch.float32, batch * vox, "out_dist", in_u8.device)
    _check_out(out_idx, torch.int32, batch * vox * ndim, "out_idx", in_u8.device)
    shape = (ctypes.c_int64 * ndim)(*spatial)
    samp = None
    if sampling is not None:
        samp = (ctypes.c_double * ndim)(*[float(s) for s in sampling])
    with torch.cuda.device(in_u8.device):
        st = _stream_handle(stream)
        rc = load().tm_dt_bf(_ptr(in_u8), ndim, shape, batch, int(metric), samp, _ptr(out_dist),
                             _ptr(out_idx), ctypes.c_void_p(st))
    if rc != TM_OK:
        raise TMError(rc, "tm_dt_bf")


def tm_edt_signed(in_u8: torch.Tensor, ndim: int, out_dist, stream=None) -> None:
    """Calls tm_edt_signed (EDT(M) - EDT(not M), unit sampling, float32)."""
    _check_mask(in_u8)
    spatial, batch = _shape_args(in_u8, ndim)
    vox = in_u8.numel() // max(batch, 1)
    _check_out(out_dist, torch.float32, batch * vox, "out_dist", in_u8.device)
    shape = (ctypes.c_int64 * ndim)(*spatial)
    with torch.cuda.device(in_u8.device):
        st = _stream_handle(stream)
        rc = load().tm_edt_signed(_ptr(in_u8), ndim, shape, batch, _ptr(out_dist), ctypes.c_void_p(st))
    if rc != TM_OK:
        raise TMError(rc, "tm_edt_signed")


def tm_cdt(in_u8: torch.Tensor, ndim: int, metric: int, out_dist, stream=None) -> None:
    """Calls tm_cdt (chamfer transform, metric code 1 taxicab / 2 chessboard)."""
    _check_mask(in_u8)
    spatial, batch = _shape_args(in_u8, ndim)
    vox = in_u8.numel() // max(batch, 1)
    _check_out(out_dist, torch.int32, batch * vox, "out_dist", in_u8.device)
    shape = (ctypes.c_int64 * ndim)(*spatial)
    with torch.cuda.device(in_u8.device):
        st = _stream_handle(stream)
        rc = load().tm_cdt(_ptr(in_u8), ndim, shape, batch, int(metric), _ptr(out_dist),
                           ctypes.c_void_p(st))
    if rc != TM_OK:
        raise TMError(rc, "tm_cdt")


def tm_cdt_workspace_size(ndim: int, spatial, batch: int, metric: int) -> int:
    """Calls tm_cdt_workspace_size: bytes of workspace tm_cdt_ws uses (0: none)."""
    shape = (ctypes.c_int64 * ndim)(*[int(v) for v in spatial])
    return int(load().tm_cdt_workspace_size(ndim, shape, int(batch), int(metric)))


def tm_cdt_ws(in_u8: torch.Tensor, ndim: int, metric: int, out_dist, workspace=None, stream=None) -> None:
    """Calls tm_cdt_ws: tm_cdt with ``workspace`` (a device tensor or None) for
    the dispatch order of its column pass."""
    _check_mask(in_u8)
    spatial, batch = _shape_args(in_u8, ndim)
    vox = in_u8.numel() // max(batch, 1)
    _check_out(out_dist, torch.int32, batch * vox, "out_dist", in_u8.device)
    nbytes = 0
    if workspace is not None:
        if workspace.device != in_u8.device or not workspace.is_contiguous():
            raise ValueError("workspace must be a contiguous tensor on %s" % in_u8.device)
        nbytes = workspace.numel() * workspace.element_size()
    shape = (ctypes.c_int64 * ndim)(*spatial)
    with torch.cuda.device(in_u8.device):
        st = _stream_handle(stream)
        rc = load().tm_cdt_ws(_ptr(in_u8), ndim, shape, batch, int(metric), _ptr(out_dist), _ptr(workspace),
                              nbytes, ctypes.c_void_p(st))
    if rc != TM_OK:
        raise TMError(rc, "tm_cdt_ws")


def _normalise_sampling(sampling, ndim):
    if sampling is None:
        return None
    if isinstance(sampling, (int, float)):
        return [float(sampling)] * ndim
    s = [float(x) for x in sampling]
    if len(s) != ndim:
        raise RuntimeError("sequence argument must have length equal to input rank")
    return s


# tm_dtype codes of the foreground predicate, by torch element type
_DTYPES = {
    torch.uint8: 0, torch.int8: 0, torch.bool: 0,
    torch.int16: 1, torch.int32: 2, torch.int64: 3,
    torch.float16: 4, torch.bfloat16: 5, torch.float32: 6, torch.float64: 7,
}
for _name in ("uint16", "uint32", "uint64"):
    if hasattr(torch, _name):
        _DTYPES[getattr(torch, _name)] = {"uint16": 1, "uint32": 2, "uint64": 3}[_name]
# 1-byte floats with a negative zero ignore the sign bit; the "fnuz" formats
# have no negative zero (0x80 is their NaN), so every nonzero byte counts
for _name, _code in (("float8_e4m3fn", 8), ("float8_e5m2", 8), ("float8_e4m3fnuz", 0),
                     ("float8_e5m2fnuz", 0)):
    if hasattr(torch, _name):
        _DTYPES[getattr(torch, _name)] = _code


def tm_mask_nonzero(x: torch.Tensor, out_u8: torch.Tensor, stream=None) -> None:
    """Calls tm_mask_nonzero: ``out_u8`` (contiguous, x.numel() bytes) gets 1
    where ``x`` is nonzero (NaN included, -0.0 excluded), read through x's strides."""
    if not x.is_cuda:
        raise ValueError("input must be a ROCm (cuda) tensor")
    if x.dtype not in _DTYPES:
        raise TypeError("input dtype %s has no nonzero test here" % x.dtype)
    _check_out(out_u8, torch.uint8, x.numel(), "out_u8", x.device)
    nd = max(x.dim(), 1)
    shape = (ctypes.c_int64 * nd)(*(x.shape if x.dim() else (1,)))
    strides = (ctypes.c_int64 * nd)(*[st * x.element_size() for st in (x.stride() if x.dim() else (1,))])
    with torch.cuda.device(x.device):
        st = _stream_handle(stream)
        rc = load().tm_mask_nonzero(_ptr(x), _DTYPES[x.dtype], nd, shape, strides, _ptr(out_u8),
                                    ctypes.c_void_p(st))
    if rc != TM_OK:
        raise TMError(rc, "tm_mask_nonzero")


def _as_mask(input: torch.Tensor) -> torch.Tensor:
    """The contiguous byte mask of ``input``: uint8 / bool contiguous tensors are
    used as they are; any other dtype or layout goes through tm_mask_nonzero."""
    if input.dtype not in _DTYPES:
        raise TypeError("input dtype %s has no nonzero test here" % input.dtype)
    if not input.is_cuda:
        raise ValueError("input must be a ROCm (cuda) tensor")
    if input.dtype in (torch.uint8, torch.bool) and input.is_contiguous():
        return input.view(torch.uint8)
    mask = torch.empty(input.shape, dtype=torch.uint8, device=input.device)
    tm_mask_nonzero(input, mask)
    return mask


def _out_buffer(given, shape, dtype, dev, what):
    """(buffer the library writes, tensor to copy it into afterwards or None).
    A pre-allocated output of the right shape and dtype is written directly
    when it is contiguous, else through a contiguous buffer (scipy fills
    any layout)."""
    if given is None:
        return torch.empty(shape, dtype=dtype, device=dev), None
    if tuple(given.shape) != tuple(shape) or given.dtype != dtype:
        raise RuntimeError("%s array has wrong shape or type" % what)
    if given.device != dev:
        raise RuntimeError("%s array is on %s, the input on %s" % (what, given.device, dev))
    if given.is_contiguous():
        return given, None
    return torch.empty(shape, dtype=dtype, device=dev), given


def distance_transform_edt(input: torch.Tensor, sampling=None, return_distances: bool = True,
                           return_indices: bool = False, distances=None, indices=None):
    """``scipy.ndimage.distance_transform_edt`` over a (B, C, *spatial) batch.

    ``input`` may have any element type and any strides: nonzero elements
    (NaN included) are foreground, as in scipy; anything but a contiguous
    uint8 / bool tensor is turned into the byte mask by tm_mask_nonzero.
    Returns float32 distances (B, C, *S) and/or int32 indices (B, C, len(S), *S),
    like scipy (a tuple when both are requested).  Pre-allocated ``distances`` /
    ``indices`` (any strides) are filled in place and not returned.  Distances
    are float32.
    """
    if input.dim() < 3:
        raise ValueError("input must be (B, C, *spatial) with 1 to 8 spatial dimensions")
    ndim = input.dim() - 2
    if ndim > 8:
        raise ValueError("at most 8 spatial dimensions are supported")
    if not (return_distances or return_indices):
        raise RuntimeError("at least one of return_distances/return_indices must be True")
    samp = _normalise_sampling(sampling, ndim)
    mask = _as_mask(input)
    lead = tuple(mask.shape[:2])
    spatial = tuple(mask.shape[2:])
    dev = mask.device
    dist_out = dist_back = idx_out = idx_back = None
    if return_distances:
        dist_out, dist_back = _out_buffer(distances, mask.shape, torch.float32, dev, "distances")
    if return_indices:
        idx_out, idx_back = _out_buffer(indices, lead + (ndim,) + spatial, torch.int32, dev, "indices")
    batch = int(lead[0]) * int(lead[1])
    ws = _workspace(dev, tm_edt_workspace_size(ndim, spatial, batch, samp, return_indices))
    tm_edt_ws(mask, ndim, samp, dist_out, idx_out, ws)
    if dist_back is not None:
        dist_back.copy_(dist_out)
    if idx_back is not None:
        idx_back.copy_(idx_out)
    result = []
    if return_distances and distances is None:
        result.append(dist_out)
    if return_indices and indices is None:
        result.append(idx_out)
    if not result:
        return None
    return result[0] if len(result) == 1 else tuple(result)


def distance_transform_bf(input: torch.Tensor, metric: str = "euclidean", sampling=None,
                          return_distances: bool = True, return_indices: bool = False):
    """``scipy.ndimage.distance_transform_bf``-style brute-force transform of a
    (B, C, *spatial) batch under "euclidean", "taxicab" or "chessboard"
    (sampling applies to every metric).  Returns float32 distances and/or
    int32 indices (B, C, len(S), *S)."""
    if input.dim() < 3:
        raise ValueError("input must be (B, C, *spatial) with 1 to 8 spatial dimensions")
    ndim = input.dim() - 2
    if not (return_distances or return_indices):
        raise RuntimeError("at least one of return_distances/return_indices must be True")
    if metric not in METRICS:
        raise ValueError("metric must be one of %s" % sorted(METRICS))
    samp = _normalise_sampling(sampling, ndim)
    mask = _as_mask(input)
    dev = mask.device
    dist = torch.empty(mask.shape, dtype=torch.float32, device=dev) if return_distances else None
    idx = None
    if return_indices:
        idx = torch.empty(tuple(mask.shape[:2]) + (ndim,) + tuple(mask.shape[2:]),
                          dtype=torch.int32, device=dev)
    tm_dt_bf(mask, ndim, METRICS[metric], samp, dist, idx)
    if dist is not None and idx is not None:
        return dist, idx
    return dist if dist is not None else idx


def distance_transform_cdt(input: torch.Tensor, metric: str = "chessboard", distances=None):
    """``scipy.ndimage.distance_transform_cdt`` over a (B, C, *spatial) batch
    for metric "chessboard" or "taxicab": int32 distances, -1 throughout a
    sample with no background.  A pre-allocated ``distances`` is filled in
    place and not returned."""
    if input.dim() < 3:
        raise ValueError("input must be (B, C, *spatial) with 1 to 8 spatial dimensions")
    ndim = input.dim() - 2
    if metric not in ("chessboard", "taxicab"):
        raise ValueError("metric must be 'chessboard' or 'taxicab'")
    mask = _as_mask(input)
    out, back = _out_buffer(distances, mask.shape, torch.int32, mask.device, "distances")
    batch = int(mask.shape[0]) * int(mask.shape[1])
    ws = _workspace(mask.device, tm_cdt_workspace_size(ndim, tuple(mask.shape[2:]), batch, METRICS[metric]))
    tm_cdt_ws(mask, ndim, METRICS[metric], out, ws)
    if back is not None:
        back.copy_(out)
    return None if distances is not None else out


def signed_distance_transform(input: torch.Tensor, distances=None):
    """EDT(M) - EDT(not M) of a (B, C, *spatial) batch: positive distance to
    the background on foreground elements, minus the distance to the
    foreground on background elements (float32, unit sampling).  A
    pre-allocated ``distances`` is filled in place and not returned."""
    if input.dim() < 3:
        raise ValueError("input must be (B, C, *spatial) with 1 to 8 spatial dimensions")
    ndim = input.dim() - 2
    mask = _as_mask(input)
    out, back = _out_buffer(distances, mask.shape, torch.float32, mask.device, "distances")
    tm_edt_signed(mask, ndim, out)
    if back is not None:
        back.copy_(out)
    return None if distances is not None else out


def distance_transform_edt_sq(input: torch.Tensor, return_indices: bool = False):
    """Exact int32 squared distances (unit sampling) of a (B, C, *spatial) batch."""
    if input.dim() < 3:
        raise ValueError("input must be (B, C, *spatial)")
    ndim = input.dim() - 2
    mask = _as_mask(input)
    sq = torch.empty(mask.shape, dtype=torch.int32, device=mask.device)
    idx = None
    if return_indices:
        idx = torch.empty(tuple(mask.shape[:2]) + (ndim,) + tuple(mask.shape[2:]),
                          dtype=torch.int32, device=mask.device)
    tm_edt_sq(mask, ndim, sq, idx)
    return (sq, idx) if return_indices else sq


def prof_enable(max_kernels: int) -> None:
    rc = load().tm_prof_enable(int(max_kernels))
    if rc != TM_OK:
        raise TMError(rc, "tm_prof_enable")


def prof_launches() -> list:
    """[(kernel name, {workgroups, threads, lds_dynamic, lds_static, regs, scratch})]
    for every kernel timed since prof_enable."""
    lib = load()
    out = []
    keys = ("workgroups", "threads", "lds_dynamic", "lds_static", "regs", "scratch")
    for i in range(lib.tm_prof_count()):
        name = ctypes.c_char_p()
        rc = lib.tm_prof_read(i, ctypes.byref(name), None)
        info = (ctypes.c_int64 * 6)()
        rc = rc or lib.tm_prof_launch(i, info)
        if rc != TM_OK:
            raise TMError(rc, "tm_prof_launch")
        out.append((name.value.decode(), dict(zip(keys, list(info)))))
    return out


def prof_read() -> list:
    """[(kernel name, ms)] for every kernel timed since prof_enable (stream must be synced)."""
    lib = load()
    out = []
    for i in range(lib.tm_prof_count()):
        name = ctypes.c_char_p()
        ms = ctypes.c_float()
        rc = lib.tm_prof_read(i, ctypes.byref(name), ctypes.byref(ms))
        if rc != TM_OK:
            raise TMError(rc, "tm_prof_read")
        out.append((name.value.decode(), float(ms.value)))
    return out
