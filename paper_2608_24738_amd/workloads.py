"""Seeded synthetic masks for the EDT, brute-force and chamfer workloads.

This module only draws inputs: it holds none of the distance-transform
arithmetic, and both the GPU tests and the CPU oracle's checks take their
masks from here.  Masks are uint8 arrays shaped (B, C, *spatial) with
nonzero = foreground, C = 1.

Every sample b of workload k draws from numpy's PCG64 seeded with
``[260824738, k, b]``.  Voxel centres sit at integer coordinates, ball
centres are continuous U[0, n_a) per axis, radii continuous U[r_min, r_max],
and a voxel is inside a ball iff sum_a (i_a - c_a)^2 <= r^2.

The paper's own benchmark masks are not described beyond their sizes, so
these shapes, densities and structures stand in for them:

  1  2-D  1x1x64x64,        foreground iff U < 0.9                 (dist + idx)
  2  2-D  32x1x512x512,     background = union of 20 discs,
                            r ~ U[5, 60]                           (dist)
  3  3-D  8x1x128^3,        foreground = union of 30 balls,
                            r ~ U[4, 30]                           (dist, exact d^2)
  4  3-D  2x1x256^3,        background iff U < 0.01,
                            sampling (2.5, 0.8, 0.8)               (dist + idx)
  5  4-D  4x1x32x64x64x64,  background iff U < 1e-4, at least one
                            background voxel per sample            (dist)

and, for the brute-force and chamfer transforms the paper also times on 2-D
batches:

  6  2-D  8x1x256x256,      background iff U < 0.01, at least one  (brute force)
  7  2-D  8x1x1024x1024,    background = union of 20 discs,
                            r ~ U[10, 120]                         (chamfer)
  8  2-D  8x1x256x256,      background = union of 20 discs,
                            r ~ U[2.5, 30]                         (chamfer)
  9  2-D  8x1x1024x1024,    as 7                                   (EDT, dist)
 10  2-D  8x1x256x256,      as 8                                   (EDT, dist)
 11  3-D  8x1x64^3,         as 3 with r ~ U[2, 15]                 (EDT, dist)
 12  3-D  2x1x256^3,        the masks and sampling of 4            (EDT, dist only)
 13  3-D  2x1x256^3,        as 3 with r ~ U[8, 60]                 (EDT, dist)
 14  2-D  8x1x1024x1024,    one background pixel per image         (EDT, dist)
 15  3-D  2x1x256^3,        one background voxel, at the origin    (EDT, dist)

Smaller twins keep the generator and scale ball radii with the smallest
extent, so parity tests can cover the same structure at sizes the oracle
finishes in seconds.
"""
from __future__ import annotations

import hashlib
from dataclasses import dataclass, field

import numpy as np

SEED = 260824738


@dataclass(frozen=True)
class Workload:
    key: int
    name: str
    batch: int
    spatial: tuple
    kind: str                    # "bernoulli_fg", "discs_bg", "balls_fg", "bernoulli_bg"
    param: dict = field(default_factory=dict)
    sampling: tuple | None = None
    want_idx: bool = False
    seed_key: int | None = None      # draw the masks of another workload (default: this one)

    @property
    def ndim(self) -> int:
        return len(self.spatial)

    @property
    def voxels(self) -> int:
        return int(self.batch * np.prod(self.spatial, dtype=np.int64))


WORKLOADS = {
    1: Workload(1, "edt2d_1x64x64_bernoulli", 1, (64, 64), "bernoulli_fg",
                {"p_fg": 0.9}, None, True),
    2: Workload(2, "edt2d_32x512x512_discs", 32, (512, 512), "discs_bg",
                {"count": 20, "r_min": 5.0, "r_max": 60.0}),
    3: Workload(3, "edt3d_8x128x128x128_balls", 8, (128, 128, 128), "balls_fg",
                {"count": 30, "r_min": 4.0, "r_max": 30.0}),
    4: Workload(4, "edt3d_2x256x256x256_aniso", 2, (256, 256, 256), "bernoulli_bg",
                {"p_bg": 0.01, "at_least_one": False}, (2.5, 0.8, 0.8), True),
    5: Workload(5, "edt4d_4x32x64x64x64_sparse", 4, (32, 64, 64, 64), "bernoulli_bg",
                {"p_bg": 1e-4, "at_least_one": True}),
    # the other transforms the paper times on 2-D batches (its throughput table)
    6: Workload(6, "bf2d_8x256x256_bernoulli1pct", 8, (256, 256), "bernoulli_bg",
                {"p_bg": 0.01, "at_least_one": True}),
    7: Workload(7, "cdt2d_8x1024x1024_discs", 8, (1024, 1024), "discs_bg",
                {"count": 20, "r_min": 10.0, "r_max": 120.0}),
    8: Workload(8, "cdt2d_8x256x256_discs", 8, (256, 256), "discs_bg",
                {"count": 20, "r_min": 2.5, "r_max": 30.0}),
    9: Workload(9, "edt2d_8x1024x1024_discs", 8, (1024, 1024), "discs_bg",
                {"count": 20, "r_min": 10.0, "r_max": 120.0}),
    10: Workload(10, "edt2d_8x256x256_discs", 8, (256, 256), "discs_bg",
                 {"count": 20, "r_min": 2.5, "r_max": 30.0}),
    11: Workload(11, "edt3d_8x64x64x64_balls", 8, (64, 64, 64), "balls_fg",
                 {"count": 30, "r_min": 2.0, "r_max": 15.0}),
    # workload 4's masks and sampling, distances only
    12: Workload(12, "edt3d_2x256x256x256_aniso_dist", 2, (256, 256, 256), "bernoulli_bg",
                 {"p_bg": 0.01, "at_least_one": False}, (2.5, 0.8, 0.8), False, seed_key=4),
    # a 3-D shape off the 128^3 / 64^3 plane path: the headline structure at 256^3
    13: Workload(13, "edt3d_2x256x256x256_balls", 2, (256, 256, 256), "balls_fg",
                 {"count": 30, "r_min": 8.0, "r_max": 60.0}),
    # the longest distances a sample can have: one background element per
    # sample (uniform position), and one at the origin corner
    14: Workload(14, "edt2d_8x1024x1024_single", 8, (1024, 1024), "single_bg", {}),
    15: Workload(15, "edt3d_2x256x256x256_corner", 2, (256, 256, 256), "corner_bg", {}),
}


def _balls(rng, spatial, count, r_min, r_max, scale):
    """Boolean union of `count` solid balls with continuous centres and radii."""
    out = np.zeros(spatial, dtype=bool)
    nd = len(spatial)
    for _ in range(count):
        c = np.array([rng.uniform(0.0, n) for n in spatial])
        r = rng.uniform(r_min, r_max) * scale
        lo = [max(0, int(np.floor(c[a] - r))) for a in range(nd)]
        hi = [min(spatial[a], int(np.ceil(c[a] + r)) + 1) for a in range(nd)]
        if any(h <= l for l, h in zip(lo, hi)):
            continue
        grids = np.ogrid[tuple(slice(l, h) for l, h in zip(lo, hi))]
        d2 = sum((g - c[a]) ** 2 for a, g in enumerate(grids))
        region = tuple(slice(l, h) for l, h in zip(lo, hi))
        out[region] |= d2 <= r * r
    return out


def sample_mask(w: Workload, b: int, spatial=None) -> np.ndarray:
    """Mask of sample `b` (uint8, nonzero = foreground) at `spatial` (default: full size)."""
    spatial = tuple(w.spatial if spatial is None else spatial)
    rng = np.random.default_rng([SEED, w.key if w.seed_key is None else w.seed_key, b])
    scale = min(spatial) / min(w.spatial)
    if w.kind == "bernoulli_fg":
        fg = rng.random(spatial) < w.param["p_fg"]
    elif w.kind == "bernoulli_bg":
        bg = rng.random(spatial) < w.param["p_bg"]
        if w.param.get("at_least_one") and not bg.any():
            pos = tuple(int(rng.integers(0, n)) for n in spatial)
            bg[pos] = True
        fg = ~bg
    elif w.kind == "discs_bg":
        fg = ~_balls(rng, spatial, w.param["count"], w.param["r_min"], w.param["r_max"], scale)
    elif w.kind == "balls_fg":
        fg = _balls(rng, spatial, w.param["count"], w.param["r_min"], w.param["r_max"], scale)
    elif w.kind == "single_bg":
        fg = np.ones(spatial, dtype=bool)
        fg[tuple(int(rng.integers(0, n)) for n in spatial)] = False
    elif w.kind == "corner_bg":
        fg = np.ones(spatial, dtype=bool)
        fg[(0,) * len(spatial)] = False
    else:
        raise ValueError(w.kind)
    return fg.astype(np.uint8)


def make_mask(key: int, spatial=None, batch=None) -> np.ndarray:
    """(B, 1, *spatial) uint8 mask of workload `key`, optionally at a smaller size."""
    w = WORKLOADS[key]
    spatial = tuple(w.spatial if spatial is None else spatial)
    batch = w.batch if batch is None else int(batch)
    out = np.empty((batch, 1) + spatial, dtype=np.uint8)
    for b in range(batch):
        out[b, 0] = sample_mask(w, b, spatial)
    return out


def mask_digest(mask: np.ndarray) -> str:
    return hashlib.sha256(np.ascontiguousarray(mask).tobytes()).hexdigest()
