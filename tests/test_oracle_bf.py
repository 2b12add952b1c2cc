"""Pins of the brute-force oracle (three metrics).  None of them re-types the
oracle: closed forms, a hand-worked fixture, the separately pinned exact
Euclidean oracle (a different algorithm), invariants of distance fields, and
scipy.ndimage as a black box where it is installed.  Planted mistakes in a
copy of the oracle must each fail one of these pins."""
import json
import os
import shutil

import numpy as np
import pytest

from oracle import edt_oracle

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
METRICS = ("euclidean", "taxicab", "chessboard")


def rand_mask(shape, p_bg, seed):
    rng = np.random.default_rng(seed)
    return (rng.random(shape) >= p_bg).astype(np.uint8)


def metric_value(metric, d, s):
    d = np.abs(np.asarray(d, np.float64))
    s = np.asarray(s, np.float64)
    if metric == "euclidean":
        return (s * s * d * d).sum(0)
    if metric == "taxicab":
        return (s * d).sum(0)
    return (s * d).max(0)


# ---- pins: each takes an oracle and raises on a mismatch ---------------------
def pin_golden_metrics(orc):
    g = json.load(open(os.path.join(GOLDEN, "metrics_two_zeros_3x4.json")))
    m = np.array(g["mask"], np.uint8)[None]
    for met in ("taxicab", "chessboard"):
        r = orc.dt_bf(m, 2, met)
        assert np.array_equal(r["value"][0], np.array(g[met], np.float64)), met
        assert np.array_equal(r["idx"][0], np.array(g[met + "_idx"])), met


def pin_single_zero(orc):
    shape, c = (5, 7, 6), (3, 1, 4)
    m = np.ones((1,) + shape, np.uint8)
    m[(0,) + c] = 0
    grid = np.indices(shape)
    for metric in METRICS:
        for sampling in (None, (1.5, 0.5, 2.0)):
            s = (1.0, 1.0, 1.0) if sampling is None else sampling
            r = orc.dt_bf(m, 3, metric, sampling)
            want = metric_value(metric, grid - np.array(c).reshape(3, 1, 1, 1),
                                np.array(s).reshape(3, 1, 1, 1))
            assert np.allclose(r["value"][0], want, rtol=1e-15, atol=0), (metric, sampling)
            assert np.all(r["idx"][0] == np.array(c).reshape(3, 1, 1, 1))


def pin_half_space(orc):
    shape, k, s0 = (6, 5), 2, 1.75
    m = np.ones((1,) + shape, np.uint8)
    m[0, :k] = 0
    x0 = np.arange(shape[0])[:, None] * np.ones(shape)
    d = np.where(x0 < k, 0.0, s0 * (x0 - k + 1))
    for metric in METRICS:
        r = orc.dt_bf(m, 2, metric, (s0, 0.5))
        want = d * d if metric == "euclidean" else d
        assert np.allclose(r["value"][0], want, rtol=1e-15, atol=0), metric


def pin_no_background(orc):
    m = np.ones((1, 3, 4), np.uint8)
    grid = np.indices((3, 4))
    for met in METRICS:
        r = orc.dt_bf(m, 2, met)
        want = metric_value(met, grid - np.array([-1, 0]).reshape(2, 1, 1), np.ones((2, 1, 1)))
        assert np.array_equal(r["value"][0], want), met
        assert np.all(r["idx"][0, 0] == -1) and np.all(r["idx"][0, 1] == 0)


def pin_exact_transform(orc, cases=6):
    for seed in range(cases):
        rng = np.random.default_rng(seed)
        nd = int(rng.integers(1, 4))
        shape = tuple(int(v) for v in rng.integers(1, 9, nd))
        m = rand_mask((2,) + shape, float(rng.uniform(0.02, 0.6)), seed)
        r = orc.dt_bf(m, nd, "euclidean")
        e = edt_oracle.edt(m, nd, None)
        assert np.array_equal(r["value"], e["sqd"]), seed
        assert np.array_equal(r["idx"], e["idx"]), seed
        samp = tuple(float(v) for v in rng.uniform(0.3, 2.5, nd))
        rs = orc.dt_bf(m, nd, "euclidean", samp)
        es = edt_oracle.edt(m, nd, samp)
        assert np.allclose(rs["value"], es["sqd"], rtol=1e-12, atol=1e-12), seed


def pin_invariants(orc, cases=4):
    shape = (7, 9, 5)
    s = np.array([1.0, 1.0, 1.0])
    grid = np.indices(shape)
    for seed in range(cases):
        m = rand_mask((1,) + shape, 0.08, seed)
        m[0, 0, 0, 0] = 0
        vals = {}
        for met in METRICS:
            r = orc.dt_bf(m, 3, met)
            v = r["value"][0]
            dist = np.sqrt(v) if met == "euclidean" else v
            vals[met] = dist
            assert np.array_equal(dist == 0, m[0] == 0)                 # zero on background
            for a in range(3):                                         # 1-Lipschitz
                assert np.all(np.abs(np.diff(dist, axis=a)) <= s[a] + 1e-12)
            idx = r["idx"][0]                                          # index: background at that value
            assert np.all(m[0][tuple(idx)] == 0)
            assert np.array_equal(metric_value(met, grid - idx, s.reshape(3, 1, 1, 1)), v)
            m2 = m.copy()                                              # monotone in the background
            m2[0, 3, 4, 2] = 0
            assert np.all(orc.dt_bf(m2, 3, met)["value"][0] <= v)
        assert np.all(vals["chessboard"] <= vals["euclidean"] + 1e-12)
        assert np.all(vals["euclidean"] <= vals["taxicab"] + 1e-12)
        assert np.all(vals["taxicab"] <= 3 * vals["chessboard"])


def pin_ties_smallest_flat(orc):
    # two zeros equidistant from the middle column under every metric
    m = np.ones((1, 3, 5), np.uint8)
    m[0, 1, 0] = 0
    m[0, 1, 4] = 0
    for met in METRICS:
        idx = orc.dt_bf(m, 2, met)["idx"][0]
        assert idx[1, 1, 2] == 0, met                                  # flat 5 beats flat 9


BF_PINS = [pin_golden_metrics, pin_single_zero, pin_half_space, pin_no_background,
           pin_exact_transform, pin_invariants, pin_ties_smallest_flat]


@pytest.mark.parametrize("pin", BF_PINS, ids=[p.__name__ for p in BF_PINS])
def test_bf_oracle_pin(pin):
    pin(edt_oracle.default())


@pytest.mark.parametrize("metric", METRICS)
def test_scipy_black_box(metric):
    ndi = pytest.importorskip("scipy.ndimage")
    cases = [((9, 11), None), ((6, 7, 5), None)]
    if metric == "euclidean":
        # scipy applies `sampling` to the euclidean metric only (observed: its
        # taxicab and chessboard results ignore it)
        cases.append(((8, 9), (1.5, 0.75)))
    for seed, (shape, samp) in enumerate(cases):
        m = rand_mask((1,) + shape, 0.1, seed)
        m[(0,) + (0,) * len(shape)] = 0
        r = edt_oracle.dt_bf(m, len(shape), metric, samp)
        d = ndi.distance_transform_bf(m[0], metric=metric, sampling=samp)
        assert np.allclose(r["dist"][0].astype(np.float64), d.astype(np.float64),
                           rtol=1e-6, atol=1e-6), (metric, shape)
        if samp is None and metric != "euclidean":
            c = ndi.distance_transform_cdt(m[0], metric=metric)
            assert np.array_equal(r["value"][0], c.astype(np.float64)), (metric, shape)


# ---- planted mistakes ------------------------------------------------------------
ORACLE_DIR = os.path.dirname(os.path.abspath(edt_oracle.__file__))
SRC = os.path.join(ORACLE_DIR, "edt_oracle.c")
BF_MUTANTS = [
    ("bf_square_dropped", "v += s[a] * s[a] * d * d;", "v += s[a] * s[a] * d;"),
    ("bf_taxicab_weight", "v += s[a] * d;", "v += d;"),
    ("bf_chessboard_sum", "else if (s[a] * d > v)\n                        v = s[a] * d;",
     "else\n                        v += s[a] * d;"),
    ("bf_ties_last", "if (v < best) {", "if (v <= best) {"),
    ("bf_virtual", "zc[0] = -1;", "zc[0] = 0;"),
    ("bf_decode_order", "zc[nz * ndim + a] = r % shape[a];\n                r /= shape[a];",
     "zc[nz * ndim + (ndim - 1 - a)] = r % shape[a];\n                r /= shape[a];"),
]


@pytest.mark.parametrize("name,old,new", BF_MUTANTS, ids=[m[0] for m in BF_MUTANTS])
def test_bf_planted_mistake_is_caught(tmp_path, name, old, new):
    text = open(SRC).read()
    assert text.count(old) == 1, "mutation anchor not found: %s" % name
    src = tmp_path / "edt_oracle.c"
    src.write_text(text.replace(old, new))
    shutil.copy(os.path.join(ORACLE_DIR, "edt_oracle.h"), tmp_path / "edt_oracle.h")
    so = edt_oracle.build(force=True, src=str(src), out=str(tmp_path / ("lib_%s.so" % name)),
                          extra=("-w",))
    orc = edt_oracle.Oracle(so)
    failed = []
    for pin in BF_PINS:
        try:
            pin(orc)
        except Exception:
            failed.append(pin.__name__)
    assert failed, "planted mistake %s passed every pin" % name
