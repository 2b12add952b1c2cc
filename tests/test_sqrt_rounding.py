"""The distance kernels round sqrt of an exact integer squared distance with
a hardware estimate and a residual correction: the estimate y is replaced by
its lower neighbour y- when x - y- * y <= 0 and by its upper neighbour y+ when
x - y+ * y > 0.  This checks, for every integer 0 < x < 2^24, that the rule
returns the correctly rounded float whenever the estimate is within one unit
in the last place of the correctly rounded value (either side).  The residual
signs are evaluated exactly in float64 (24-bit by 24-bit products fit)."""
import numpy as np


def corrected(y, x):
    yb = y.view(np.uint32)
    ym = (yb - np.uint32(1)).view(np.float32).astype(np.float64)
    yp = (yb + np.uint32(1)).view(np.float32).astype(np.float64)
    yd = y.astype(np.float64)
    r = np.where(x - ym * yd <= 0, ym, yd)
    r = np.where(x - yp * yd > 0, yp, r)
    return r.astype(np.float32)


def test_residual_correction_is_exact_for_all_24_bit_integers():
    x = np.arange(1, 1 << 24, dtype=np.float64)
    # float64 sqrt then float32 rounding is the correctly rounded float32
    # sqrt (53 >= 2 * 24 + 2, so the double rounding is innocuous)
    rn = np.sqrt(x).astype(np.float32)
    rb = rn.view(np.uint32)
    for shift in (-1, 0, 1):
        y = (rb.astype(np.int64) + shift).astype(np.uint32).view(np.float32)
        got = corrected(y, x)
        bad = np.flatnonzero(got.view(np.uint32) != rb)
        assert bad.size == 0, (shift, x[bad[:5]])
