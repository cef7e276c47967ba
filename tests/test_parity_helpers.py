"""The comparison rules of the GPU parity tests, exercised on the CPU with
planted differences (the rules themselves must accept what the tolerances
allow and reject everything else)."""
import numpy as np
import pytest

import _parity as PT


def _codes(seed=0, n=2, dk=8, dv=6):
    rng = np.random.default_rng(seed)
    y = rng.uniform(-7, 7, (n, dk, dv))
    return np.rint(y).astype(np.int8), y


def test_compare_codes_rules():
    c, y = _codes()
    assert PT.compare_codes(c.copy(), c, y, frac=1.0) == 0
    g = c.copy()
    y2 = y.copy()
    y2[0, 1, 2] = 2.5005                          # a tie within the window
    c2 = np.rint(y2).astype(np.int8)
    g = c2.copy()
    g[0, 1, 2] = 2                                # other rounding of the tie
    assert PT.compare_codes(g, c2, y2, frac=1.0) == 1
    with pytest.raises(AssertionError):           # too many for the fraction
        PT.compare_codes(g, c2, y2, frac=0.0)
    g2 = c.copy()
    g2[1, 0, 0] += 1                              # away from a tie
    y3 = y.copy()
    y3[1, 0, 0] = np.floor(y3[1, 0, 0]) + 0.2
    c3 = np.rint(y3).astype(np.int8)
    g3 = c3.copy()
    g3[1, 0, 0] += 1
    with pytest.raises(AssertionError):
        PT.compare_codes(g3, c3, y3, frac=1.0)
    g4 = c2.copy()
    g4[0, 1, 2] += 2                              # two levels
    with pytest.raises(AssertionError):
        PT.compare_codes(g4, c2, y2, frac=1.0)


def test_compare_refit_rules():
    c, y = _codes(1)
    n, dk, dv = c.shape
    r = np.full((n, dk), 0.5, np.float32)
    cc = np.full((n, dv), 2.0, np.float32)
    lo = cc.astype(np.float64) * 0.999
    hi = cc.astype(np.float64) * 1.001
    bits = np.full((n, dk), 4, np.uint8)          # q_b = 7
    nb, _ = PT.compare_refit(c.copy(), r.copy(), cc.copy(), c, r, cc, y, (lo, hi), bits, frac=1.0)
    assert nb == 0
    g_c = cc.copy()
    g_c[0, 3] = cc[0, 3] * 1.01                   # outside the admissible range
    with pytest.raises(AssertionError):
        PT.compare_refit(c.copy(), r.copy(), g_c, c, r, cc, y, (lo, hi), bits, frac=1.0)
    g_r = r.copy()
    g_r[1, 2] *= 1 + 1e-4                         # row scale beyond SCALE_REL
    with pytest.raises(AssertionError):
        PT.compare_refit(c.copy(), g_r, cc.copy(), c, r, cc, y, (lo, hi), bits, frac=1.0)
    # an admissible column shift: the GPU's codes are the rounding of y under
    # its own scale, which here moves one code to the next level
    y2 = y.copy()
    y2[0, 4, 3] = 5.4980
    c2 = np.rint(y2).astype(np.int8)
    g_c = cc.copy()
    g_c[0, 3] = cc[0, 3] / 1.0008                 # y scales by 1.0008 -> 5.5024 -> 6
    g = c2.copy()
    g[0, 4, 3] = 6
    nb, _ = PT.compare_refit(g, r.copy(), g_c, c2, r, cc, y2, (lo, hi), bits, frac=1.0)
    assert nb == 1
    with pytest.raises(AssertionError):           # keeping the oracle's code is wrong under that scale
        PT.compare_refit(c2.copy(), r.copy(), g_c, c2, r, cc, y2, (lo, hi), bits, frac=0.0)
    g[0, 4, 3] = 7                                # two levels: never
    with pytest.raises(AssertionError):
        PT.compare_refit(g, r.copy(), g_c, c2, r, cc, y2, (lo, hi), bits, frac=1.0)


def test_compare_out_rules():
    o = np.linspace(-2, 2, 50)
    PT.compare_out(o + 1e-3 * np.abs(o) * 0.9, o)
    with pytest.raises(AssertionError):
        PT.compare_out(o + 2e-3 * np.abs(o) + 1e-4, o)


def test_compare_pivots_rules():
    rng = np.random.default_rng(3)
    X = rng.standard_normal((2, 5, 8)) * 0.3
    mask = np.zeros((2, 5), bool)
    mask[0, 1] = mask[1, 3] = True
    o_pv = X.astype(np.float16).view(np.uint16)
    assert PT.compare_pivots(o_pv.copy(), o_pv, X, mask, frac=1.0) == 0
    g = o_pv.copy()
    g[0, 1, 2] += 1                                  # one binary16 step away from the rounding of X
    X2 = X.copy()
    X2[0, 1, 2] = (g[0, 1, 2:3].view(np.float16).astype(np.float64)[0]
                   + o_pv[0, 1, 2:3].view(np.float16).astype(np.float64)[0]) / 2    # exactly between: a tie
    assert PT.compare_pivots(g, o_pv, X2, mask, frac=1.0) == 1
    with pytest.raises(AssertionError):            # not a tie: the value is wrong
        PT.compare_pivots(g, o_pv, X, mask, frac=1.0)
    g2 = o_pv.copy()
    g2[0, 2, 0] += 7                                 # outside the pivot rows: not compared
    assert PT.compare_pivots(g2, o_pv, X, mask, frac=0.0) == 0
