"""Properties every exact EDT result must satisfy, at any size.

Used on the oracle (against its pins) and on GPU results at sizes where the
oracle cannot be run element by element.  Nothing here computes a transform.
"""
import numpy as np


def check_index_valid(mask, sq, idx, sampling=None, rtol=0.0, atol=0.0):
    """idx(x) is a background element at squared distance sq(x) from x.

    mask (*S) nonzero = foreground; sq (*S); idx (nd, *S).  With no background
    in the sample, idx must be the virtual element (-1, 0, ..., 0).
    Returns the number of violating elements (0 = valid).
    """
    mask = np.asarray(mask)
    shape = mask.shape
    nd = len(shape)
    idx = np.asarray(idx).astype(np.int64)
    sq = np.asarray(sq)
    w = (np.ones(nd) if sampling is None
         else np.broadcast_to(np.asarray(sampling, np.float64), (nd,)) ** 2)
    grid = np.indices(shape, dtype=np.int64)
    if not (mask == 0).any():
        virt = np.zeros(nd, np.int64)
        virt[0] = -1
        bad = np.zeros(shape, bool)
        for a in range(nd):
            bad |= idx[a] != virt[a]
    else:
        inside = np.ones(shape, bool)
        for a in range(nd):
            inside &= (idx[a] >= 0) & (idx[a] < shape[a])
        clipped = tuple(np.clip(idx[a], 0, shape[a] - 1) for a in range(nd))
        bad = ~inside | (mask[clipped] != 0)
    # distance realised by idx
    diff2 = [(grid[a] - idx[a]) ** 2 for a in range(nd)]
    if sampling is None and np.issubdtype(sq.dtype, np.integer):
        real = sum(diff2)
        bad |= real != sq
    else:
        real = sum(w[a] * diff2[a] for a in range(nd))
        bad |= np.abs(real - sq) > atol + rtol * np.abs(sq)
    return int(bad.sum())


def check_zero_iff_background(mask, dist):
    """dist == 0 exactly on background (only when the sample has background)."""
    mask = np.asarray(mask)
    if not (mask == 0).any():
        return int((np.asarray(dist) == 0).sum())
    return int(((np.asarray(dist) == 0) != (mask == 0)).sum())


def check_lipschitz(dist, sampling=None, slack=0.0):
    """|D(x) - D(x + e_a)| <= s_a along every axis.  Returns violations."""
    dist = np.asarray(dist, np.float64)
    nd = dist.ndim
    s = (np.ones(nd) if sampling is None
         else np.broadcast_to(np.asarray(sampling, np.float64), (nd,)))
    bad = 0
    for a in range(nd):
        if dist.shape[a] < 2:
            continue
        step = np.abs(np.diff(dist, axis=a))
        bad += int((step > s[a] * (1 + slack) + slack).sum())
    return bad


def chamfer_fixed_point_violations(mask, d, metric):
    """Number of elements where d breaks the chamfer equations on one sample.

    With N(x) the face neighbours (taxicab) or all 3^nd - 1 neighbours
    (chessboard) inside the grid, the graph distance D to the background is
    the only integer field with D = 0 on the background and
    D(x) = 1 + min over N(x) of D elsewhere (follow a shortest path for <=,
    a chain of neighbours whose value drops by one for >=), and on the full
    grid it equals the taxicab or chessboard distance.  A sample without
    background must hold -1 everywhere.
    """
    mask = np.asarray(mask)
    d = np.asarray(d).astype(np.int64)
    if not (mask == 0).any():
        return int((d != -1).sum())
    nd = mask.ndim
    big = np.int64(1) << 40
    pad = np.pad(d, 1, constant_values=big)
    if metric == "taxicab":
        offs = []
        for a in range(nd):
            for s in (-1, 1):
                o = [0] * nd
                o[a] = s
                offs.append(o)
    else:
        offs = [o for o in np.ndindex(*(3,) * nd)]
        offs = [[v - 1 for v in o] for o in offs if any(v != 1 for v in o)]
    nb = np.full(d.shape, big)
    for o in offs:
        sl = tuple(slice(1 + oa, 1 + oa + n) for oa, n in zip(o, d.shape))
        nb = np.minimum(nb, pad[sl])
    want = np.where(mask == 0, 0, nb + 1)
    return int((d != want).sum() + (d < 0).sum())
