"""Pins for the CPU oracle: facts fixed by the paper or by mathematics.

Each function takes a loaded oracle (``oracle.edt_oracle.Oracle``) and raises
AssertionError on the first disagreement.  They are run against the real
oracle, and against copies with planted mistakes to show that each mistake
is caught (test_oracle_mutants.py).

Pins (none of them re-types the oracle's own formula):
  * all-pairs brute force on tiny random masks (the definition, by numpy);
  * hand-worked fixtures under tests/golden/;
  * closed forms: one background element, a background half-space,
    all background, no background (virtual element);
  * the 1-D textbook nearest-zero scan;
  * invariants: index validity, zero iff background, 1-Lipschitz,
    monotonicity under added background, flip / permutation equivariance,
    batch = per sample.
"""
import glob
import json
import os

import numpy as np

from bruteforce import brute_force
from invariants import check_index_valid, check_lipschitz, check_zero_iff_background

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def tiny_cases(seed=0, count=160, max_rank=4, max_extent=6):
    """Random tiny masks: ranks 1..max_rank, extents 1..max_extent, mixed densities."""
    rng = np.random.default_rng(seed)
    dens = [0.0, 0.05, 0.2, 0.5, 0.8, 0.95, 1.0]
    out = []
    for c in range(count):
        nd = 1 + c % max_rank
        shape = tuple(int(rng.integers(1, max_extent + 1)) for _ in range(nd))
        p_bg = dens[c % len(dens)]
        mask = (rng.random(shape) >= p_bg).astype(np.uint8)
        out.append(mask)
    return out


def pin_bruteforce_unit(orc, count=160):
    for mask in tiny_cases(1, count):
        r = orc.edt(mask[None])
        sq, idx = brute_force(mask)
        assert np.array_equal(r["sq"][0], sq), ("sq", mask.shape)
        assert np.array_equal(r["idx"][0], idx), ("idx", mask.shape)
        assert np.array_equal(r["sqd"][0], sq.astype(np.float64))
        assert np.array_equal(r["dist"][0], np.sqrt(sq.astype(np.float64)).astype(np.float32))


def pin_bruteforce_sampled(orc, count=120):
    rng = np.random.default_rng(7)
    for mask in tiny_cases(2, count):
        nd = mask.ndim
        samp = tuple(float(x) for x in rng.uniform(0.3, 3.0, nd))
        r = orc.edt(mask[None], sampling=samp)
        sq, _ = brute_force(mask, samp)
        assert np.allclose(r["sqd"][0], sq, rtol=1e-12, atol=1e-12), (mask.shape, samp)
        assert check_index_valid(mask, r["sqd"][0], r["idx"][0], samp, rtol=1e-12, atol=1e-12) == 0
        assert np.allclose(r["dist"][0], np.sqrt(sq), rtol=1e-6, atol=1e-7)


def pin_bruteforce_sampled_exact(orc, count=120):
    """Sampling 2.0 on every axis keeps all double arithmetic exact, so the
    sampled path must give 4x the unit result and the same canonical index."""
    for mask in tiny_cases(3, count):
        nd = mask.ndim
        r = orc.edt(mask[None], sampling=(2.0,) * nd)
        sq, idx = brute_force(mask)
        assert np.array_equal(r["sqd"][0], 4.0 * sq), mask.shape
        assert np.array_equal(r["idx"][0], idx), mask.shape


def pin_golden(orc):
    files = sorted(glob.glob(os.path.join(GOLDEN, "*.json")))
    assert files
    files = [fn for fn in files if "sq" in json.load(open(fn))]   # Euclidean fixtures
    assert files
    for fn in files:
        g = json.load(open(fn))
        mask = np.asarray(g["mask"], np.uint8).reshape(g["shape"])
        r = orc.edt(mask[None], sampling=g["sampling"])
        want_sq = np.asarray(g["sq"]).reshape(g["shape"])
        got = r["sq"][0] if g["sampling"] is None else r["sqd"][0]
        assert np.array_equal(got, want_sq), os.path.basename(fn)
        assert np.array_equal(r["idx"][0], np.asarray(g["idx"])), os.path.basename(fn)


def pin_single_zero(orc):
    """One background element c: D2(x) = sum_a w_a (x_a - c_a)^2, idx = c."""
    rng = np.random.default_rng(11)
    for trial in range(24):
        nd = 1 + trial % 4
        shape = tuple(int(rng.integers(1, 9 if nd < 4 else 6)) for _ in range(nd))
        c = tuple(int(rng.integers(0, n)) for n in shape)
        mask = np.ones(shape, np.uint8)
        mask[c] = 0
        grid = np.indices(shape, dtype=np.int64)
        want = sum((grid[a] - c[a]) ** 2 for a in range(nd))
        r = orc.edt(mask[None])
        assert np.array_equal(r["sq"][0], want)
        for a in range(nd):
            assert np.all(r["idx"][0][a] == c[a])
        samp = tuple(float(x) for x in rng.uniform(0.5, 2.5, nd))
        want_s = sum(samp[a] ** 2 * (grid[a] - c[a]) ** 2 for a in range(nd))
        r = orc.edt(mask[None], sampling=samp)
        assert np.allclose(r["sqd"][0], want_s, rtol=1e-13, atol=0)


def pin_halfspace(orc):
    """Background = {x_a < k} along one axis a: D(x) = s_a (x_a - k + 1) for x_a >= k,
    and the nearest element is x with x_a replaced by k - 1."""
    for nd, shape in [(1, (9,)), (2, (7, 5)), (3, (4, 6, 5)), (4, (3, 4, 2, 5))]:
        for a in range(nd):
            for k in range(1, shape[a]):
                mask = np.ones(shape, np.uint8)
                sl = [slice(None)] * nd
                sl[a] = slice(0, k)
                mask[tuple(sl)] = 0
                grid = np.indices(shape, dtype=np.int64)
                dd = np.maximum(grid[a] - (k - 1), 0)
                r = orc.edt(mask[None])
                assert np.array_equal(r["sq"][0], dd * dd), (shape, a, k)
                want_idx = grid.copy()
                want_idx[a] = np.minimum(grid[a], k - 1)
                assert np.array_equal(r["idx"][0], want_idx), (shape, a, k)
                s = 1.7
                samp = [1.0] * nd
                samp[a] = s
                r = orc.edt(mask[None], sampling=samp)
                assert np.allclose(r["sqd"][0], (s * dd) ** 2, rtol=1e-14, atol=0)


def _scan_1d(mask):
    """Textbook nearest-zero scan: last zero on the left, first on the right."""
    n = len(mask)
    left = [-1] * n
    last = None
    for x in range(n):
        if mask[x] == 0:
            last = x
        left[x] = last
    right = [None] * n
    nxt = None
    for x in range(n - 1, -1, -1):
        if mask[x] == 0:
            nxt = x
        right[x] = nxt
    sq, idx = [], []
    for x in range(n):
        cands = [y for y in (left[x], right[x]) if y is not None]
        if not cands:
            sq.append((x + 1) ** 2)
            idx.append(-1)
            continue
        y = min(cands, key=lambda y: (abs(x - y), y))
        sq.append((x - y) ** 2)
        idx.append(y)
    return np.array(sq), np.array(idx)


def pin_textbook_1d(orc):
    rng = np.random.default_rng(5)
    for trial in range(60):
        n = int(rng.integers(1, 40))
        mask = (rng.random(n) >= rng.choice([0.02, 0.1, 0.3, 0.7])).astype(np.uint8)
        sq, idx = _scan_1d(mask)
        r = orc.edt(mask[None])
        assert np.array_equal(r["sq"][0], sq), mask
        assert np.array_equal(r["idx"][0][0], idx), mask


def pin_all_background_and_none(orc):
    for shape in [(1,), (5,), (3, 4), (2, 3, 4), (2, 2, 3, 2)]:
        nd = len(shape)
        zero = np.zeros(shape, np.uint8)
        r = orc.edt(zero[None])
        assert np.all(r["sq"][0] == 0) and np.all(r["dist"][0] == 0)
        assert np.array_equal(r["idx"][0], np.indices(shape))
        one = np.ones(shape, np.uint8)
        grid = np.indices(shape, dtype=np.int64)
        want = (grid[0] + 1) ** 2 + sum(grid[a] ** 2 for a in range(1, nd))
        r = orc.edt(one[None])
        assert np.array_equal(r["sq"][0], want), shape
        assert np.all(r["idx"][0][0] == -1)
        for a in range(1, nd):
            assert np.all(r["idx"][0][a] == 0)


def pin_invariants(orc):
    rng = np.random.default_rng(13)
    for trial in range(30):
        nd = 1 + trial % 4
        shape = tuple(int(rng.integers(2, 14 if nd <= 2 else 7)) for _ in range(nd))
        mask = (rng.random(shape) >= rng.choice([0.05, 0.3, 0.6])).astype(np.uint8)
        samp = tuple(float(x) for x in rng.uniform(0.5, 2.0, nd))
        r = orc.edt(mask[None])
        sq, dist, idx = r["sq"][0], r["dist"][0], r["idx"][0]
        assert check_index_valid(mask, sq, idx) == 0
        assert check_zero_iff_background(mask, dist) == 0
        assert check_lipschitz(dist, slack=1e-6) == 0
        rs = orc.edt(mask[None], sampling=samp)
        assert check_index_valid(mask, rs["sqd"][0], rs["idx"][0], samp, 1e-12, 1e-12) == 0
        assert check_lipschitz(rs["dist"][0], samp, slack=1e-6) == 0
        # monotone: adding background never increases the distance (once the
        # sample has background; the virtual element can be nearer than a new one)
        if (mask == 0).any():
            more = mask.copy()
            more[tuple(int(rng.integers(0, n)) for n in shape)] = 0
            r2 = orc.edt(more[None])
            assert np.all(r2["sq"][0] <= sq)
        # flips and axis permutations commute with the transform (not with the
        # virtual element of a sample without background)
        if not (mask == 0).any():
            continue
        ax = int(rng.integers(0, nd))
        rf = orc.edt(np.flip(mask, ax)[None])
        assert np.array_equal(rf["sq"][0], np.flip(sq, ax))
        perm = tuple(rng.permutation(nd))
        rp = orc.edt(np.transpose(mask, perm)[None])
        assert np.array_equal(rp["sq"][0], np.transpose(sq, perm))
        rps = orc.edt(np.transpose(mask, perm)[None], sampling=tuple(samp[p] for p in perm))
        assert np.allclose(rps["sqd"][0], np.transpose(rs["sqd"][0], perm), rtol=1e-12, atol=1e-12)
    # batch == per sample
    masks = np.stack([(rng.random((6, 5, 4)) >= p).astype(np.uint8) for p in (0.0, 0.1, 0.5, 1.0)])
    rb = orc.edt(masks, ndim=3)
    for b in range(len(masks)):
        r1 = orc.edt(masks[b][None])
        assert np.array_equal(rb["sq"][b], r1["sq"][0])
        assert np.array_equal(rb["idx"][b], r1["idx"][0])


ALL_PINS = [pin_bruteforce_unit, pin_bruteforce_sampled, pin_bruteforce_sampled_exact,
            pin_golden, pin_single_zero, pin_halfspace, pin_textbook_1d,
            pin_all_background_and_none, pin_invariants]
