"""Pins for the calibration side of the oracle (oracle/calibration.py):
row-impact factors, candidate-format distortions, lifetime weights, the
allocators and the pivot choice, each against an independent form."""
import itertools
import math

import numpy as np
import pytest

import oracle
import oracle.calibration as CAL


def _stream(seed, T=40, H=3, dk=6, kda=False):
    rng = np.random.default_rng(seed)
    q = rng.standard_normal((T, H, dk)); q /= np.linalg.norm(q, axis=-1, keepdims=True)
    k = rng.standard_normal((T, H, dk)); k /= np.linalg.norm(k, axis=-1, keepdims=True)
    beta = rng.uniform(0, 1, (T, H))
    gate = rng.uniform(0.6, 1.0, (T, H, dk)) if kda else rng.uniform(0.6, 1.0, (T, H))
    return q, k, beta, gate


@pytest.mark.parametrize("kda", [False, True])
def test_row_impact_is_mean_square_of_transported_query(kda):
    """omega_i = mean_t ((A_t^T q_t)_i)^2 with A_t = (I - beta k k^T) D formed as
    a matrix here (Proposition 1, Appendix A.2); w has geometric mean 1 per
    head and w_i / w_j = (omega_i / omega_j)^{gamma/2} (Section 4.3 footnote)."""
    q, k, beta, gate = _stream(1, kda=kda)
    T, H, dk = q.shape
    w, omega = CAL.row_impact(q, k, beta, gate, gamma=0.25)
    ref = np.zeros((H, dk))
    for t in range(T):
        for h in range(H):
            D = np.diag(gate[t, h] if kda else np.full(dk, gate[t, h]))
            A = (np.eye(dk) - beta[t, h] * np.outer(k[t, h], k[t, h])) @ D
            ref[h] += (A.T @ q[t, h]) ** 2
    np.testing.assert_allclose(omega, ref / T, rtol=1e-12)
    np.testing.assert_allclose(np.exp(np.log(w).mean(axis=1)), 1.0, rtol=1e-12)
    np.testing.assert_allclose(w[:, 0] / w[:, 1], (omega[:, 0] / omega[:, 1]) ** 0.125, rtol=1e-12)


def test_fit_dual_axis_column_fit_and_start():
    """The codec's column factor is the weighted least-squares solve for the
    codes fixed at the absmax start (library solve), and that start puts each
    column's largest |X|/r on the top level."""
    rng = np.random.default_rng(2)
    n, dk, dv = 3, 10, 7
    X = rng.standard_normal((n, dk, dv)) * np.exp(rng.standard_normal((n, dk, 1)))
    bits = rng.choice([2, 4, 8], size=(n, dk)).astype(np.uint8)
    w = np.exp(0.4 * rng.standard_normal((n, dk)))
    codes, r, c = oracle.fit_dual_axis(X, bits, w=w)
    np.testing.assert_allclose(r.astype(np.float64) ** 2 * w, np.abs(X).mean(axis=2), rtol=2.5e-7)
    qb = (2.0 ** (bits.astype(np.int64) - 1) - 1)[:, :, None]
    rr = r.astype(np.float64)[:, :, None]
    c0 = (np.abs(X) / rr).max(axis=1)
    z = np.clip(np.rint(X * qb / (rr * c0[:, None, :])), -qb, qb) / qb
    for t in range(n):
        for j in range(dv):
            A = (w[t] * rr[t, :, 0] * z[t, :, j])[:, None]
            sol = np.linalg.lstsq(A, w[t] * X[t, :, j], rcond=None)[0][0]
            assert abs(float(c[t, j]) - sol) <= 1e-7 * abs(sol)
    assert np.array_equal(codes, oracle.quantize(X, r, c, bits))


def test_distortion_units_and_binary16():
    """b = 16 is the binary16 rounding error (numpy's IEEE half); per-head
    distortion is the w^2-weighted mean of the per-row ones; wider codes cost
    less on these states."""
    rng = np.random.default_rng(3)
    C, H, dk, dv = 4, 2, 8, 16
    S = rng.standard_normal((C, H, dk, dv)) * 0.1
    w = np.exp(0.3 * rng.standard_normal((H, dk)))
    cands = [2, 4, 8, 16]
    d_row = CAL.calib_distortion(S, cands, "row", w=w)
    d_head = CAL.calib_distortion(S, cands, "head", w=w)
    e16 = ((S.astype(np.float16).astype(np.float64) - S) ** 2).mean(axis=(0, 3)).reshape(-1)
    np.testing.assert_allclose(d_row[:, 3], e16, rtol=1e-12)
    np.testing.assert_allclose(d_head, (d_row.reshape(H, dk, 4) * w[:, :, None] ** 2).mean(axis=1), rtol=1e-12)
    assert np.all(d_row[:, 0] > d_row[:, 1]) and np.all(d_row[:, 1] > d_row[:, 2]) and np.all(d_row[:, 2] > d_row[:, 3])


def test_distortion_pivots_leave_the_column_fit():
    """With pivot rows the integer rows' distortion equals that of the state
    without the pivot rows, however large the pivots (Appendix A.3)."""
    rng = np.random.default_rng(4)
    C, H, dk, dv = 3, 2, 9, 8
    S = rng.standard_normal((C, H, dk, dv)) * 0.1
    piv = np.zeros((H, dk), bool)
    piv[0, 2] = piv[1, 5] = piv[1, 7] = True
    S[:, piv, :] *= 1e3
    d = CAL.calib_distortion(S, [4, 8], "row", pivots=piv).reshape(H, dk, 2)
    for h in range(H):
        keep = ~piv[h]
        d_h = CAL.calib_distortion(S[:, h:h + 1, keep], [4, 8], "row").reshape(-1, 2)
        np.testing.assert_array_equal(d[h, keep], d_h)


def test_lifetime_weight_is_a_geometric_series():
    ell = np.array([-0.3, -0.01, -1e-4, 0.0])
    L = CAL.lifetime_weights(ell, 64)
    ref = [(1 - math.exp(2 * 64 * e)) / (1 - math.exp(2 * e)) if e != 0 else 64.0 for e in ell]
    np.testing.assert_allclose(L, ref, rtol=1e-10)


def test_dp_allocation_is_exact():
    """Dynamic programming equals exhaustive enumeration of Eq. 6 on small
    random instances (unequal unit sizes, several budgets)."""
    rng = np.random.default_rng(5)
    cands = [2, 4, 8]
    for trial in range(40):
        U = int(rng.integers(1, 6))
        n_u = rng.choice([64, 128], size=U)
        cost = np.sort(rng.uniform(0, 1, (U, 3)), axis=1)[:, ::-1] * rng.uniform(0.1, 10, (U, 1))
        budget = float(rng.choice([2.0, 3.0, 4.0, 5.5, 6.0, 8.0]))
        bf = CAL.allocate_bruteforce(cost, n_u, cands, budget)
        dp = CAL.allocate_dp(cost, n_u, cands, budget)
        vbf = sum(cost[u, bf[u]] for u in range(U))
        vdp = sum(cost[u, dp[u]] for u in range(U))
        assert abs(vbf - vdp) <= 1e-12 * max(1.0, vbf)
        assert sum(n_u[u] * cands[dp[u]] for u in range(U)) <= budget * n_u.sum() + 1e-9


def test_lagrangian_allocation_properties():
    """Lagrangian with repair: within budget; never better than the exact
    optimum; no single upgrade that fits is left; and an assignment of the
    multiplier alone is optimal for the budget it spends (the Lagrangian
    sufficiency condition)."""
    rng = np.random.default_rng(6)
    cands = [2, 4, 8]
    for trial in range(30):
        U = int(rng.integers(2, 7))
        n_u = np.full(U, 128)
        cost = np.sort(rng.uniform(0, 1, (U, 3)), axis=1)[:, ::-1] * rng.uniform(0.1, 10, (U, 1))
        budget = float(rng.choice([3.0, 4.0, 5.0, 6.0]))
        lg = CAL.allocate_lagrangian(cost, n_u, cands, budget)
        dp = CAL.allocate_dp(cost, n_u, cands, budget)
        spent = sum(n_u[u] * cands[lg[u]] for u in range(U))
        assert spent <= budget * n_u.sum() + 1e-9
        assert sum(cost[u, lg[u]] for u in range(U)) >= sum(cost[u, dp[u]] for u in range(U)) - 1e-12
        left = budget * n_u.sum() - spent
        for u in range(U):
            for ci in range(3):
                extra = n_u[u] * (cands[ci] - cands[lg[u]])
                if 0 < extra <= left:
                    assert cost[u, ci] >= cost[u, lg[u]]
        lam = float(rng.uniform(0, 0.05))
        pure = np.array([min(range(3), key=lambda ci: (cost[u, ci] + lam * n_u[u] * cands[ci], cands[ci]))
                         for u in range(U)])
        b_star = sum(n_u[u] * cands[pure[u]] for u in range(U)) / n_u.sum()
        opt = CAL.allocate_dp(cost, n_u, cands, b_star)
        assert abs(sum(cost[u, pure[u]] for u in range(U)) - sum(cost[u, opt[u]] for u in range(U))) <= 1e-12


def test_pivot_choice_is_top_risk():
    rng = np.random.default_rng(7)
    risk = rng.uniform(0, 1, 50)
    risk[[3, 9]] = risk[4]                        # ties go to the lower index
    m = CAL.select_pivots(risk, 7)
    assert m.sum() == 7 and np.min(risk[m]) >= np.max(risk[~m])


def test_mean_log_retention_units_closed_forms():
    """l_u (Appendix A.3) of the oracle: gates a^t over T samples give
    log(a) (T - 1) / 2 for every unit; a scalar gate gives each of its
    head's rows the head's value; a head's value is the mean of its rows'."""
    import math
    import oracle.calibration as CAL
    T, H, dk = 6, 2, 5
    a = np.array([0.9, 0.5])
    g = np.stack([a ** t for t in range(T)])                     # [T][H]
    rows = CAL.mean_log_retention_units(g, dk, "row").reshape(H, dk)
    np.testing.assert_allclose(rows, np.log(a)[:, None] * (T - 1) / 2 * np.ones((1, dk)), rtol=1e-13)
    np.testing.assert_allclose(CAL.mean_log_retention_units(g, dk, "head"), np.log(a) * (T - 1) / 2, rtol=1e-13)
    rng = np.random.default_rng(3)
    gk = rng.uniform(0.2, 1.0, (T, H, dk))
    r = CAL.mean_log_retention_units(gk, dk, "row").reshape(H, dk)
    assert math.isclose(r[1, 3], sum(math.log(gk[t, 1, 3]) for t in range(T)) / T, rel_tol=1e-13)
    np.testing.assert_allclose(CAL.mean_log_retention_units(gk, dk, "head"), r.mean(axis=1), rtol=1e-13)
