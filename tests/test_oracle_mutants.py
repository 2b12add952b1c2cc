"""Each plausible mistake planted in a copy of the oracle fails at least one pin.

The copy is patched textually, compiled with gcc into a temporary directory
and run through the same pins as the real oracle (CPU only).
"""
import os
import shutil

import pytest

import pins
from oracle import edt_oracle

ORACLE_DIR = os.path.dirname(os.path.abspath(edt_oracle.__file__))
SRC = os.path.join(ORACLE_DIR, "edt_oracle.c")

# (name, text in edt_oracle.c, planted replacement).
# Not listed: popping on "<" instead of "<=".  That change is equivalent: a
# parabola kept with a one-point interval is never selected, because a query
# only moves to the next parabola when its interval starts strictly before
# the query position, so no output can tell the two rules apart.
MUTANTS = [
    ("query_nonstrict", "(__int128)zn[j + 1] < (__int128)q * zd[j + 1]",
     "(__int128)zn[j + 1] <= (__int128)q * zd[j + 1]"),
    ("dropped_square", "num = (f[q] + q * q) - (f[p] + p * p);",
     "num = (f[q] + q) - (f[p] + p * p);"),
    ("wrong_sign", "den = 2 * (q - p);", "den = 2 * (p - q);"),
    ("axis_order", "for (int axis = ndim - 1; axis >= 0 && rc == 0; --axis)",
     "for (int axis = 0; axis < ndim && rc == 0; ++axis)"),
    ("virtual_point", "y[0] = -1;", "y[0] = 0;"),
    ("query_wrong_operand", "g[q] = f[p] + (q - p) * (q - p);",
     "g[q] = f[q] + (q - p) * (q - p);"),
    ("line_base", "int64_t base = o * n * inner + i;", "int64_t base = o * n + i;"),
    ("decode_order", "for (int a = ndim - 1; a >= 0; --a) {\n                    y[a] = t % shape[a];",
     "for (int a = 0; a < ndim; ++a) {\n                    y[a] = t % shape[a];"),
    ("dbl_weight_dropped", "g[q] = f[p] + w * d * d;", "g[q] = f[p] + d * d;"),
    ("dbl_den_weight", "(2.0 * w * (dq - dp));", "(2.0 * (dq - dp));"),
    ("dbl_query_nonstrict", "while (j < k && z[j + 1] < (double)q)",
     "while (j < k && z[j + 1] <= (double)q)"),
    ("skip_no_site_check", "if (f[q] == NO_SITE_I)\n            continue;", ""),
]


def fast_pins(orc):
    """All pins at reduced case counts; returns the names of those that fail."""
    failed = []
    for pin in pins.ALL_PINS:
        try:
            if pin.__name__.startswith("pin_bruteforce"):
                pin(orc, count=60)
            else:
                pin(orc)
        except Exception:
            failed.append(pin.__name__)
    return failed


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_planted_mistake_is_caught(tmp_path, name, old, new):
    text = open(SRC).read()
    assert text.count(old) == 1, "mutation anchor not found: %s" % name
    src = tmp_path / "edt_oracle.c"
    src.write_text(text.replace(old, new))
    shutil.copy(os.path.join(ORACLE_DIR, "edt_oracle.h"), tmp_path / "edt_oracle.h")
    so = edt_oracle.build(force=True, src=str(src), out=str(tmp_path / ("lib_%s.so" % name)),
                          extra=("-w",))
    failed = fast_pins(edt_oracle.Oracle(so))
    assert failed, "planted mistake %s passed every pin" % name
