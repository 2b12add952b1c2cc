"""All-pairs nearest-background search on tiny inputs (numpy, independent of the oracle).

The definition written out: D2(x) = min over background y of
sum_a w_a (x_a - y_a)^2; the index is the first minimiser in row-major order
of the background list, i.e. the smallest flat index among nearest ones.
Samples without background use the virtual element (-1, 0, ..., 0).
"""
import numpy as np


def brute_force(mask, sampling=None):
    """mask: (*spatial) array, nonzero = foreground. Returns (sq, idx) with
    sq int64 (unit sampling) or float64, idx int32 of shape (ndim, *spatial)."""
    mask = np.asarray(mask)
    shape = mask.shape
    nd = len(shape)
    unit = sampling is None or np.all(np.asarray(sampling, dtype=np.float64) == 1.0)
    coords = np.indices(shape).reshape(nd, -1).T.astype(np.int64)      # (V, nd), row-major
    zeros = coords[mask.reshape(-1) == 0]                               # row-major order
    if len(zeros) == 0:
        virt = np.zeros((1, nd), np.int64)
        virt[0, 0] = -1
        zeros = virt
    diff = coords[:, None, :] - zeros[None, :, :]                      # (V, Z, nd)
    if unit:
        cost = (diff * diff).sum(-1)
    else:
        w = np.broadcast_to(np.asarray(sampling, dtype=np.float64), (nd,)) ** 2
        cost = (w * (diff * diff)).sum(-1)
    arg = cost.argmin(axis=1)                                           # first occurrence
    sq = cost[np.arange(len(coords)), arg].reshape(shape)
    idx = zeros[arg].T.reshape((nd,) + shape).astype(np.int32)
    return sq, idx
