"""ctypes loader for the C oracle (``edt_oracle.c``) plus a numpy wrapper.

Test infrastructure only (tests, smoke check, CPU-baseline timing); it imports
nothing from the GPU library.  What the oracle computes is documented in
``edt_oracle.c``: the exact Euclidean distance transform by the separable
lower-envelope method of the paper's Section 2.3.2, in int64 arithmetic for
unit sampling and in double otherwise, and the brute-force transform under
the euclidean, taxicab and chessboard metrics.  The chamfer transform and the
point-wise spot check below are plain numpy over the brute-force values.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "edt_oracle.c")
_LIB = os.path.join(_HERE, "liboracle_edt.so")
_lock = threading.Lock()
_lib = None


def build(force: bool = True, src: str = _SRC, out: str = _LIB, extra=()) -> str:
    """Compile an oracle source with gcc (OpenMP across lines). Returns the .so path."""
    if not force and os.path.exists(out) and os.path.getmtime(out) >= os.path.getmtime(src):
        return out
    tmp = out + ".tmp%d" % os.getpid()
    cmd = ["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared", "-Wall", "-Wextra",
           "-I", _HERE, *extra, "-o", tmp, src, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


class Oracle:
    """One loaded build of the oracle library."""

    def __init__(self, path: str):
        lib = ctypes.CDLL(path)
        lib.oracle_edt.restype = ctypes.c_int
        lib.oracle_edt.argtypes = [
            ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p, ctypes.c_int64,
            ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
            ctypes.c_void_p, ctypes.c_int]
        lib.oracle_dt_bf.restype = ctypes.c_int
        lib.oracle_dt_bf.argtypes = [
            ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int,
            ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int]
        lib.oracle_threads_used.restype = ctypes.c_int
        lib.oracle_threads_used.argtypes = [ctypes.c_int]
        self.lib = lib
        self.path = path

    def threads_used(self, nthreads: int) -> int:
        return int(self.lib.oracle_threads_used(int(nthreads)))

    def edt(self, mask: np.ndarray, ndim: int | None = None, sampling=None, *,
            want_sq: bool = True, want_dist: bool = True, want_idx: bool = True,
            nthreads: int = 1) -> dict:
        """Exact EDT of ``mask`` with shape (batch..., *spatial) (nonzero = foreground).

        ``ndim`` defaults to ``mask.ndim - 1``; leading axes before the spatial
        ones are folded into the batch.  Returns a dict with
          ``sq``   int64 exact squared distance (unit sampling only, else None),
          ``sqd``  float64 squared distance,
          ``dist`` float32 distance (sqrt correctly rounded),
          ``idx``  int32 coordinates, shape (batch..., ndim, *spatial),
        each None when not requested.
        """
        mask = np.ascontiguousarray(mask)
        if mask.dtype != np.uint8:
            mask = (mask != 0).astype(np.uint8)
        if ndim is None:
            ndim = mask.ndim - 1
        lead = mask.shape[:mask.ndim - ndim]
        spatial = tuple(int(s) for s in mask.shape[mask.ndim - ndim:])
        batch = int(np.prod(lead, dtype=np.int64))
        vox = int(np.prod(spatial, dtype=np.int64))
        unit = is_unit(sampling, ndim)
        samp = None
        if not unit:
            samp = np.ascontiguousarray(
                np.broadcast_to(np.asarray(sampling, dtype=np.float64), (ndim,)))
        shape = np.asarray(spatial, dtype=np.int64)
        sq = np.empty((batch, vox), np.int64) if (want_sq and unit) else None
        sqd = np.empty((batch, vox), np.float64) if want_sq else None
        dist = np.empty((batch, vox), np.float32) if want_dist else None
        idx = np.empty((batch, ndim, vox), np.int32) if want_idx else None
        rc = self.lib.oracle_edt(_ptr(mask), ndim, _ptr(shape), batch, _ptr(samp),
                                 _ptr(sq), _ptr(sqd), _ptr(dist), _ptr(idx), int(nthreads))
        if rc != 0:
            raise ValueError("oracle_edt failed with code %d" % rc)
        return {
            "sq": None if sq is None else sq.reshape(lead + spatial),
            "sqd": None if sqd is None else sqd.reshape(lead + spatial),
            "dist": None if dist is None else dist.reshape(lead + spatial),
            "idx": None if idx is None else idx.reshape(lead + (ndim,) + spatial),
        }


    def dt_bf(self, mask: np.ndarray, ndim: int | None = None, metric: str = "euclidean",
              sampling=None, *, want_idx: bool = True, nthreads: int = 1) -> dict:
        """Brute-force transform of ``mask`` (batch..., *spatial) under ``metric``
        ("euclidean", "taxicab" or "chessboard").  Returns a dict with
          ``value`` float64 metric value (euclidean: the squared distance),
          ``dist``  float32 distance (euclidean: sqrt of the value, correctly
                    rounded; the others: the value),
          ``idx``   int32 coordinates (batch..., ndim, *spatial) or None."""
        mask = np.ascontiguousarray(mask)
        if mask.dtype != np.uint8:
            mask = (mask != 0).astype(np.uint8)
        if ndim is None:
            ndim = mask.ndim - 1
        code = METRICS[metric]
        lead = mask.shape[:mask.ndim - ndim]
        spatial = tuple(int(s) for s in mask.shape[mask.ndim - ndim:])
        batch = int(np.prod(lead, dtype=np.int64))
        vox = int(np.prod(spatial, dtype=np.int64))
        samp = None
        if sampling is not None:
            samp = np.ascontiguousarray(
                np.broadcast_to(np.asarray(sampling, dtype=np.float64), (ndim,)))
        shape = np.asarray(spatial, dtype=np.int64)
        value = np.empty((batch, vox), np.float64)
        idx = np.empty((batch, ndim, vox), np.int32) if want_idx else None
        rc = self.lib.oracle_dt_bf(_ptr(mask), ndim, _ptr(shape), batch, code, _ptr(samp),
                                   _ptr(value), _ptr(idx), int(nthreads))
        if rc != 0:
            raise ValueError("oracle_dt_bf failed with code %d" % rc)
        dist = (np.sqrt(value) if code == 0 else value).astype(np.float32)
        return {
            "value": value.reshape(lead + spatial),
            "dist": dist.reshape(lead + spatial),
            "idx": None if idx is None else idx.reshape(lead + (ndim,) + spatial),
        }


    def cdt(self, mask: np.ndarray, ndim: int | None = None, metric: str = "chessboard", *,
            nthreads: int = 1) -> np.ndarray:
        """Chamfer transform (paper, Section 2.3.2; Table 1 lists it as exact):
        for metric "taxicab" or "chessboard", the int32 distance from every
        element to the nearest background element of its sample, which is the
        brute-force value above, and -1 throughout a sample with no background
        (a unit-weight chamfer sweep reaches nothing there)."""
        if metric not in ("taxicab", "chessboard"):
            raise ValueError(metric)
        mask = np.ascontiguousarray(mask)
        if ndim is None:
            ndim = mask.ndim - 1
        value = self.dt_bf(mask, ndim, metric, want_idx=False, nthreads=nthreads)["value"]
        lead = mask.shape[:mask.ndim - ndim]
        flat = value.reshape(int(np.prod(lead, dtype=np.int64)), -1)
        out = flat.astype(np.int64)
        has_bg = (mask.reshape(flat.shape) == 0).any(axis=1)
        out[~has_bg] = -1
        return out.astype(np.int32).reshape(mask.shape)


def signed_edt(mask: np.ndarray, ndim: int | None = None, *, nthreads: int = 1) -> np.ndarray:
    """Signed transform EDT(M) - EDT(not M) (the distance field of boundary
    losses the paper's introduction and Section 2.3.2 motivate): the exact
    transform of the mask minus that of its complement, float32, unit
    sampling.  Exactly one of the two terms is nonzero at every element."""
    mask = np.ascontiguousarray(mask)
    inv = (mask == 0).astype(np.uint8)
    pos = edt(mask, ndim, None, want_sq=False, want_idx=False, nthreads=nthreads)["dist"]
    neg = edt(inv, ndim, None, want_sq=False, want_idx=False, nthreads=nthreads)["dist"]
    return (pos - neg).astype(np.float32)


def metric_dt_at(sample: np.ndarray, metric: str, points: np.ndarray) -> np.ndarray:
    """The metric value (euclidean: squared distance) from each of `points`
    (k x ndim integer coordinates) to the nearest background element of one
    unit-sampled sample, by visiting every background element: the definition
    of the transform, for spot checks at sizes where the whole brute-force
    transform is too slow.  NaN where the sample has no background."""
    z = np.argwhere(np.asarray(sample) == 0).astype(np.int64)
    pts = np.asarray(points, dtype=np.int64)
    out = np.full(len(pts), np.nan)
    if len(z) == 0:
        return out
    for i0 in range(0, len(pts), 64):
        d = np.abs(pts[i0:i0 + 64, None, :] - z[None, :, :])
        if metric == "euclidean":
            v = (d * d).sum(axis=2)
        elif metric == "taxicab":
            v = d.sum(axis=2)
        elif metric == "chessboard":
            v = d.max(axis=2)
        else:
            raise ValueError(metric)
        out[i0:i0 + 64] = v.min(axis=1)
    return out


METRICS = {"euclidean": 0, "taxicab": 1, "chessboard": 2}


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def is_unit(sampling, ndim: int) -> bool:
    if sampling is None:
        return True
    s = np.broadcast_to(np.asarray(sampling, dtype=np.float64), (ndim,))
    return bool(np.all(s == 1.0))


def default() -> Oracle:
    """The oracle built from ``edt_oracle.c`` (compiled on first use)."""
    global _lib
    with _lock:
        if _lib is None:
            _lib = Oracle(build(force=False))
    return _lib


def threads_used(nthreads: int) -> int:
    return default().threads_used(nthreads)


def edt(mask, ndim=None, sampling=None, **kw) -> dict:
    return default().edt(mask, ndim, sampling, **kw)


def dt_bf(mask, ndim=None, metric="euclidean", sampling=None, **kw) -> dict:
    return default().dt_bf(mask, ndim, metric, sampling, **kw)


def cdt(mask, ndim=None, metric="chessboard", **kw) -> np.ndarray:
    return default().cdt(mask, ndim, metric, **kw)
