"""Pins for the oracle's second level normalisation, N2: the stored integer
q of a b-bit row stands for the level z = 2^(8-b) q (the paper's KDA
codebook, Appendix C.1), so S^ = r c 2^(8-b) q and the largest level is
top_b = 2^(8-b) q_b (127, 112, 64 for b = 8, 4, 2).  N1 (z = q / q_b) is
pinned in test_oracle_pins.py.

Each test checks N2 against something outside the oracle: exact level
values, brute-force enumeration, exact ties, the fit's no-clip bound, a
library least-squares solve, or the identity that relates the two
normalisations on rows of one width (N2 with row factor r is N1 with row
factor r top_b).
"""
import itertools

import numpy as np
import pytest

import oracle
from test_oracle_pins import _refit_case, _unit

N2 = oracle.LEVELS_POW2


def _top(b):
    return (2 ** (b - 1) - 1) * 2.0 ** (8 - b)


@pytest.mark.parametrize("b", [2, 4, 8])
def test_pow2_levels_exact_and_idempotent(b):
    """Every code of every width reconstructs to exactly r c 2^(8-b) q and
    survives dequantize -> quantize unchanged; the extreme codes sit at
    +-r c top_b."""
    qb = 2 ** (b - 1) - 1
    rng = np.random.default_rng(100 + b)
    dk, dv = 3, 2 * qb + 1
    codes = np.tile(np.arange(-qb, qb + 1, dtype=np.int8), (dk, 1))[None]
    r = rng.uniform(0.01, 2, (1, dk)).astype(np.float32)
    c = rng.uniform(0.01, 2, (1, dv)).astype(np.float32)
    bits = np.full((1, dk), b, np.uint8)
    S = oracle.dequant(codes, r, c, bits, levels=N2)
    want = r[0].astype(np.float64)[:, None] * c[0].astype(np.float64)[None, :] * codes[0] * 2.0 ** (8 - b)
    assert np.array_equal(S[0], want)
    assert np.array_equal(oracle.quantize(S, r, c, bits, levels=N2), codes)
    np.testing.assert_allclose(np.abs(S[0, :, 0]), r[0] * np.float64(c[0, 0]) * _top(b), rtol=1e-15)


def test_pow2_bruteforce_2x2_nearest_level():
    """On 2x2 tiles the N2 codes minimise sum_i w_i^2 (X - X^)^2 over all
    joint code choices (b <= 4) and are the per-entry nearest level (b = 8)."""
    rng = np.random.default_rng(105)
    for trial in range(40):
        bits = rng.choice([2, 4, 8], size=2).astype(np.uint8)
        r = rng.uniform(0.05, 1.0, 2).astype(np.float32) / 64
        c = rng.uniform(0.05, 1.0, 2).astype(np.float32)
        X = rng.standard_normal((2, 2)) * 0.6
        w = rng.uniform(0.5, 2.0, 2)
        got = oracle.quantize(X[None], r[None], c[None], bits[None], levels=N2)[0]
        codes = [np.arange(-(2 ** (int(b) - 1) - 1), 2 ** (int(b) - 1)) for b in bits]
        step = np.array([2.0 ** (8 - int(b)) for b in bits])
        if max(bits) <= 4:
            best, best_err = None, np.inf
            for z in itertools.product(codes[0], codes[0], codes[1], codes[1]):
                Z = np.array(z, dtype=np.float64).reshape(2, 2)
                Xh = r[:, None].astype(np.float64) * c[None, :].astype(np.float64) * Z * step[:, None]
                err = np.sum(w[:, None] ** 2 * (X - Xh) ** 2)
                if err < best_err:
                    best, best_err = Z, err
            assert np.array_equal(got, best.astype(np.int8))
        for i in range(2):
            for j in range(2):
                cand = float(r[i]) * float(c[j]) * codes[i] * step[i]
                assert got[i, j] == codes[i][np.argmin(np.abs(X[i, j] - cand))]


def test_pow2_error_bound_clip_and_ties():
    """|X^ - X| <= r c 2^(8-b) / 2 where X is in range, out of range clips to
    +-q_b, and exact half-way values round to the even neighbour."""
    rng = np.random.default_rng(106)
    n, dk, dv = 4, 8, 8
    bits = rng.choice([2, 4, 8], size=(n, dk)).astype(np.uint8)
    r = rng.uniform(0.1, 1, (n, dk)).astype(np.float32) / 64
    c = rng.uniform(0.1, 1, (n, dv)).astype(np.float32)
    X = rng.standard_normal((n, dk, dv)) * 1.5
    codes, y = oracle.quantize(X, r, c, bits, want_y=True, levels=N2)
    Xh = oracle.dequant(codes, r, c, bits, levels=N2)
    qb = (2.0 ** (bits.astype(np.int64) - 1) - 1)[:, :, None]
    step = (2.0 ** (8 - bits.astype(np.int64)))[:, :, None]
    rc = r.astype(np.float64)[:, :, None] * c.astype(np.float64)[:, None, :]
    inside = np.abs(y) <= qb
    assert inside.mean() > 0.1 and (~inside).any()
    assert np.all((np.abs(Xh - X) <= rc * step / 2 * (1 + 1e-12))[np.broadcast_to(inside, X.shape)])
    assert np.all(codes[~inside] == np.sign(y[~inside]) * np.broadcast_to(qb, y.shape)[~inside])
    # ties: b = 4, r c = 1, so y = X / 16 exactly
    halfs = np.array([0.5, 1.5, 2.5, -0.5, -1.5, -6.5])
    cq, yq = oracle.quantize((16 * halfs)[None, None, :], np.full((1, 1), 0.5, np.float32),
                             np.full((1, 6), 2.0, np.float32), np.array([[4]], np.uint8), want_y=True, levels=N2)
    assert np.array_equal(yq[0, 0], halfs) and cq[0, 0].tolist() == [0, 2, 2, 0, -2, -6]


def test_pow2_fit_reaches_the_top_level():
    """The N2 setup fit keeps r_i c_j top_i >= |S_ij|, with equality (to fp32
    rounding) at each column's arg-max of |S_ij| / (r_i top_i); the codes of
    the fitted state never clip and reach +-q_b there; r is the N1 row
    factor (the level normalisation does not enter it)."""
    rng = np.random.default_rng(107)
    S = (rng.standard_normal((3, 16, 12)) * np.exp(rng.standard_normal((3, 16, 1)))).astype(np.float32)
    w = rng.uniform(0.5, 2.0, (3, 16))
    bits = rng.choice([2, 4, 8], size=(3, 16)).astype(np.uint8)
    r, c = oracle.fit_absmax(S, w, bits=bits, levels=N2)
    r1, _ = oracle.fit_absmax(S, w)
    assert np.array_equal(r, r1)
    top = np.vectorize(_top)(bits.astype(np.int64))[:, :, None]
    bound = r.astype(np.float64)[:, :, None] * c.astype(np.float64)[:, None, :] * top
    assert np.all(bound >= np.abs(S))
    np.testing.assert_allclose((np.abs(S) / bound).max(axis=1), 1.0, rtol=3e-7)
    codes, y = oracle.quantize(S.astype(np.float64), r, c, bits, want_y=True, levels=N2)
    qb = (2.0 ** (bits.astype(np.int64) - 1) - 1)[:, :, None]
    assert np.all(np.abs(y) <= qb * (1 + 1e-12))
    am = (np.abs(S) / bound).argmax(axis=1)
    hit = np.take_along_axis(np.abs(codes.astype(np.int64)), am[:, None, :], axis=1)[:, 0]
    assert np.array_equal(hit, np.take_along_axis(qb[:, :, 0], am, axis=1).astype(np.int64))
    with pytest.raises(ValueError):
        oracle.fit_absmax(S, w, levels=N2)          # the widths are needed


def _one_width(b, seed, n=3, dk=16, dv=10, kda=False):
    """A case whose rows all have width b, with row factors of at most 16
    significant bits, so that r top_b is exact in fp32."""
    codes, r, c, bits, q, k, v, g, beta, w = _refit_case(seed=seed, n=n, dk=dk, dv=dv, kda=kda)
    bits = np.full_like(bits, b)
    r2 = (np.round(r.astype(np.float64) * 2 ** 12) / 2 ** 12 / _top(b)).astype(np.float32)
    r2 = np.maximum(r2, np.float32(2.0 ** -12))
    r2 = (np.round(r2.astype(np.float64) * 2 ** 16) / 2 ** 16).astype(np.float32)
    r1 = (r2.astype(np.float64) * _top(b)).astype(np.float32)
    assert np.array_equal(r1.astype(np.float64), r2.astype(np.float64) * _top(b))
    qb = 2 ** (b - 1) - 1
    rng = np.random.default_rng(seed + 1)
    codes = rng.integers(-qb, qb + 1, size=codes.shape).astype(np.int8)
    return codes, r1, r2, c, bits, q, k, v, g, beta, w


@pytest.mark.parametrize("kda", [False, True])
@pytest.mark.parametrize("b", [2, 4, 8])
def test_pow2_is_n1_with_rescaled_rows(b, kda):
    """On rows of one width the two normalisations differ by the constant
    top_b folded into r: N2 with row factors r equals N1 with r top_b, for
    reconstruction, the frozen step, the refit (whose c' then agree and
    whose r' is normalisation-free) and the row-absmax step (whose r'
    differs by top_b)."""
    codes, r1, r2, c, bits, q, k, v, g, beta, w = _one_width(b, 110 + b, kda=kda)
    np.testing.assert_allclose(oracle.dequant(codes, r2, c, bits, levels=N2), oracle.dequant(codes, r1, c, bits),
                               rtol=1e-14, atol=0)
    n1 = oracle.decode_step(codes, r1, c, bits, q, k, v, g, beta, want_y=True)
    n2 = oracle.decode_step(codes, r2, c, bits, q, k, v, g, beta, want_y=True, levels=N2)
    assert np.array_equal(n1[0], n2[0])
    np.testing.assert_allclose(n2[1], n1[1], rtol=1e-13, atol=1e-15)
    np.testing.assert_allclose(n2[2], n1[2], rtol=1e-13, atol=1e-13)
    f1 = oracle.decode_step_refit(codes, r1, c, bits, q, k, v, g, beta, w=w)
    f2 = oracle.decode_step_refit(codes, r2, c, bits, q, k, v, g, beta, w=w, levels=N2)
    assert np.array_equal(f1[0], f2[0]) and np.array_equal(f1[1], f2[1])
    np.testing.assert_allclose(f2[2].astype(np.float64) * _top(b), f1[2], rtol=2.5e-7)
    m1 = oracle.decode_step_rowmax(codes, r1, c, bits, q, k, v, g, beta)
    m2 = oracle.decode_step_rowmax(codes, r2, c, bits, q, k, v, g, beta, levels=N2)
    assert np.array_equal(m1[0], m2[0]) and np.array_equal(m1[2], m2[2])
    np.testing.assert_allclose(m2[1].astype(np.float64) * _top(b), m1[1], rtol=2.5e-7)


@pytest.mark.parametrize("kda", [False, True])
def test_pow2_refit_on_mixed_widths(kda):
    """Mixed widths, where the normalisations genuinely differ: the absmax
    start puts each column's largest |y0_ij| / q_b at exactly 1; the column
    factor solves the weighted least squares with v_ij = r'_i 2^(8-b_i) z_ij
    (library solve); the final codes are the N2 quantizer on (r', c')."""
    codes, r, c, bits, q, k, v, g, beta, w = _refit_case(seed=120, kda=kda)
    r = r / np.float32(64)
    out, rn, cn, _, ex = oracle.decode_step_refit(codes, r, c, bits, q, k, v, g, beta, w=w, want=("X", "y0"),
                                                  levels=N2)
    qb = (2.0 ** (bits.astype(np.int64) - 1) - 1)[:, :, None]
    step = (2.0 ** (8 - bits.astype(np.int64)))[:, :, None]
    np.testing.assert_allclose((np.abs(ex["y0"]) / qb).max(axis=1), 1.0, rtol=0, atol=1e-12)
    z = np.clip(np.rint(ex["y0"]), -qb, qb) * step
    X = ex["X"]
    n, dk, dv = X.shape
    for t in range(n):
        for j in range(dv):
            A = (w[t] * rn[t].astype(np.float64) * z[t, :, j])[:, None]
            if not np.any(A):
                continue
            sol = np.linalg.lstsq(A, w[t] * X[t, :, j], rcond=None)[0][0]
            assert abs(float(cn[t, j]) - sol) <= 1e-7 * abs(sol)
    assert np.array_equal(out, oracle.quantize(X, rn, cn, bits, levels=N2))


def test_pow2_rowmax_reaches_the_top_level():
    """N2 row-absmax: r'_i = max_j |X_ij| / top_i, so every row's largest
    entry lands on +-q_b, and no entry is off by more than half a level
    r' 2^(8-b) / 2."""
    codes, r, c, bits, q, k, v, g, beta, _ = _refit_case(seed=121)
    out, rn, cn, o = oracle.decode_step_rowmax(codes, r, c, bits, q, k, v, g, beta, levels=N2)
    S = oracle.dequant(codes, r, c, bits, levels=N2)
    X, _ = oracle.update_fp(S, q, k, v, g, beta)
    top = np.vectorize(_top)(bits.astype(np.int64))
    np.testing.assert_allclose(rn, np.abs(X).max(axis=2) / top, rtol=6e-8, atol=0)
    qb = (2.0 ** (bits.astype(np.int64) - 1) - 1)
    am = np.abs(X).argmax(axis=2)
    hit = np.take_along_axis(out, am[:, :, None], axis=2)[:, :, 0]
    assert np.array_equal(np.abs(hit).astype(np.int64), qb.astype(np.int64))
    step = (2.0 ** (8 - bits.astype(np.int64)))[:, :, None]
    Xh = rn.astype(np.float64)[:, :, None] * out * step
    assert np.all(np.abs(Xh - X) <= rn.astype(np.float64)[:, :, None] * step / 2 * (1 + 1e-6))
