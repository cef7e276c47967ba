"""Oracle for the calibration side of the setup step: row-impact factors,
candidate-format distortions, lifetime weights, the bit allocators and the
FP16 pivot choice (Section 3.2, Section 4.3, Appendices A.2, A.3, C.1, C.2).

TEST INFRASTRUCTURE ONLY (see oracle/__init__.py): plain fp64 loops and
numpy, in the paper's order and notation, sharing no code with libstepq.
"""
from __future__ import annotations

import itertools
import math

import numpy as np

from . import dequant, double_to_half, fit_dual_axis, half_to_double

OMEGA_FLOOR = 2.0 ** -120


def row_impact(q, k, beta, gate, gamma: float = 0.25):
    """Row-impact factors of every head.

    omega_i = E_cal[g_i^2] with g = A^T q, A = (I - beta k k^T) D (the one-step
    readout sensitivity, Appendix A.2 with H = 1; Appendix C.1 gives the KDA
    closed form g_i = d_i (q_i - beta k_i k^T q)), then per head
    w_i = omega_i^{gamma/2} / GM_j(omega_j^{gamma/2}) (Section 4.3 footnote).
    q, k [T][H][dk]; beta [T][H]; gate [T][H] (GDN, D = alpha I) or
    [T][H][dk] (KDA).  omega is floored at 2^-120 so that a row no key or
    query ever touches still gets a finite factor.  Returns (w, omega)
    [H][dk]."""
    q, k = np.asarray(q, np.float64), np.asarray(k, np.float64)
    beta, gate = np.asarray(beta, np.float64), np.asarray(gate, np.float64)
    T, H, dk = q.shape
    omega = np.zeros((H, dk))
    for t in range(T):
        for h in range(H):
            d = gate[t, h] if gate.ndim == 3 else np.full(dk, gate[t, h])
            kq = sum(k[t, h, i] * q[t, h, i] for i in range(dk))
            for i in range(dk):
                g = d[i] * (q[t, h, i] - beta[t, h] * k[t, h, i] * kq)
                omega[h, i] += g * g
    omega /= T
    omega = np.maximum(omega, OMEGA_FLOOR)
    w = np.empty((H, dk))
    for h in range(H):
        p = omega[h] ** (gamma / 2)
        gm = math.exp(sum(math.log(x) for x in p) / dk)
        w[h] = p / gm
    return w, omega


def calib_distortion(states, cand_bits, unit: str, w=None, pivots=None):
    """Candidate-format distortion d_u(b) (Appendix A.3).

    states [C][H][dk][dv] sampled reference states; for each candidate b every
    non-pivot row of every sample is coded at width b by the spatial codec
    (the dual-axis fit, with the factors w) and reconstructed; b = 16 is the
    binary16 rounding.  unit "row" (KDA): d = unweighted MSE of the key row
    over samples and columns; unit "head" (Qwen): d = w_i^2-weighted MSE over
    the head's elements and samples.  pivots [H][dk] bool: rows held in
    binary16, left out of the column fit.  Returns [U][len(cand_bits)]."""
    S = np.asarray(states, np.float64)
    C, H, dk, dv = S.shape
    wt = np.ones((H, dk)) if w is None else np.asarray(w, np.float64)
    piv = np.zeros((H, dk), bool) if pivots is None else np.asarray(pivots, bool)
    err = np.zeros((len(cand_bits), H, dk))                 # summed squared error per row
    X = S.reshape(C * H, dk, dv)
    for ci, b in enumerate(cand_bits):
        if b == 16:
            R = half_to_double(double_to_half(X))
        else:
            bits = np.where(piv, 16, b).astype(np.uint8)
            bt = np.broadcast_to(bits[None], (C, H, dk)).reshape(C * H, dk)
            wtile = np.broadcast_to(wt[None], (C, H, dk)).reshape(C * H, dk)
            res = fit_dual_axis(X, bt, w=wtile)
            codes, r, c = res[:3]
            R = dequant(codes, r, c, bt, pv=res[3] if len(res) > 3 else None)
        e = ((R - X) ** 2).reshape(C, H, dk, dv)
        err[ci] = e.sum(axis=(0, 3))
    if unit == "row":
        return (err / (C * dv)).reshape(len(cand_bits), H * dk).T.copy()
    if unit == "head":
        return ((err * wt[None] ** 2).sum(axis=2) / (C * dk * dv)).T.copy()
    raise ValueError(unit)


def mean_log_retention_units(gates, d_k: int, unit: str):
    """l_u (Appendix A.3): mean over calibration samples of the log of the
    gate that decays the unit, gates [T][H] (head gate) or [T][H][d_k]
    (channel gate); key-row units [H*d_k] or head units [H] (the mean over
    the head's rows).  Plain loops."""
    g = np.asarray(gates, np.float64)
    T, H = g.shape[:2]
    rows = np.zeros((H, d_k))
    for h in range(H):
        for i in range(d_k):
            s = 0.0
            for t in range(T):
                s += math.log(g[t, h, i] if g.ndim == 3 else g[t, h])
            rows[h, i] = s / T
    if unit == "row":
        return rows.reshape(-1)
    return np.array([sum(rows[h]) / d_k for h in range(H)])


def lifetime_weights(ell, horizon: int):
    """L_u = sum_{j=0}^{H-1} exp(2 j l_u) (Section 3.2)."""
    return np.array([sum(math.exp(2.0 * j * e) for j in range(horizon)) for e in np.asarray(ell, np.float64)])


def allocate_bruteforce(cost, n_u, cand_bits, budget):
    """Exact minimiser of sum_u cost[u][b_u] s.t. sum_u n_u b_u <= budget
    sum_u n_u, by enumeration (tiny U only).  Ties: the first in
    lexicographic order of candidate indices.  Returns candidate indices."""
    cost = np.asarray(cost, np.float64)
    U = cost.shape[0]
    cap = budget * float(np.sum(n_u))
    best, arg = math.inf, None
    for choice in itertools.product(range(len(cand_bits)), repeat=U):
        if sum(n_u[u] * cand_bits[choice[u]] for u in range(U)) > cap + 1e-9:
            continue
        v = sum(cost[u, choice[u]] for u in range(U))
        if v < best:
            best, arg = v, choice
    return None if arg is None else np.array(arg)


def allocate_dp(cost, n_u, cand_bits, budget):
    """Multiple-choice knapsack by dynamic programming over units and spent
    bits (Appendix C.2, the Qwen optimizer): weights n_u b in units of their
    greatest common divisor.  Returns candidate indices minimising the total
    cost within the budget (None if infeasible)."""
    cost = np.asarray(cost, np.float64)
    U, nc = cost.shape
    wts = [[int(n_u[u]) * int(b) for b in cand_bits] for u in range(U)]
    g = 0
    for row in wts:
        for x in row:
            g = math.gcd(g, x)
    wts = [[x // g for x in row] for row in wts]
    cap = int(math.floor(budget * float(np.sum(n_u)) / g + 1e-9))
    INF = math.inf
    best = [0.0] + [INF] * cap                      # best[s]: min cost with exactly s spent
    choice = []
    for u in range(U):
        new = [INF] * (cap + 1)
        pick = [-1] * (cap + 1)
        for s in range(cap + 1):
            if best[s] == INF:
                continue
            for ci in range(nc):
                s2 = s + wts[u][ci]
                if s2 <= cap and best[s] + cost[u, ci] < new[s2]:
                    new[s2] = best[s] + cost[u, ci]
                    pick[s2] = ci
        choice.append(pick)
        best = new
    s_end = min(range(cap + 1), key=lambda s: (best[s], s))
    if best[s_end] == INF:
        return None
    out = np.zeros(U, int)
    s = s_end
    for u in range(U - 1, -1, -1):
        ci = choice[u][s]
        out[u] = ci
        s -= wts[u][ci]
    return out


def allocate_lagrangian(cost, n_u, cand_bits, budget, iters: int = 200):
    """Lagrangian allocation with repair (Appendix C.2, the KDA optimizer):
    each unit minimises cost[u][b] + lam n_u b for a shared multiplier lam,
    the smallest lam whose assignment fits the budget is found by bisection,
    then the remaining budget is spent by repeatedly taking the single
    upgrade (one unit to a wider candidate) with the largest cost decrease per
    extra bit that still fits.  Returns candidate indices."""
    cost = np.asarray(cost, np.float64)
    U, nc = cost.shape
    nb = np.asarray(cand_bits, np.float64)
    n_u = np.asarray(n_u, np.float64)
    cap = budget * float(np.sum(n_u))

    def assign(lam):
        out = np.zeros(U, int)
        for u in range(U):
            vals = [cost[u, ci] + lam * n_u[u] * nb[ci] for ci in range(nc)]
            out[u] = min(range(nc), key=lambda ci: (vals[ci], nb[ci]))     # ties: the narrower
        return out

    def spent(ch):
        return float(sum(n_u[u] * nb[ch[u]] for u in range(U)))

    lo, hi = 0.0, 1.0
    while spent(assign(hi)) > cap:
        hi *= 2.0
        if hi > 1e300:
            raise ValueError("budget below the narrowest assignment")
    if spent(assign(lo)) <= cap:
        ch = assign(lo)
    else:
        for _ in range(iters):
            mid = 0.5 * (lo + hi)
            if spent(assign(mid)) <= cap:
                hi = mid
            else:
                lo = mid
        ch = assign(hi)
    # repair: spend what is left on the best upgrades per bit
    while True:
        left = cap - spent(ch)
        best, arg = 0.0, None
        for u in range(U):
            for ci in range(nc):
                extra = n_u[u] * (nb[ci] - nb[ch[u]])
                if extra <= 0 or extra > left + 1e-9:
                    continue
                gain = (cost[u, ch[u]] - cost[u, ci]) / extra
                if gain > best:
                    best, arg = gain, (u, ci)
        if arg is None:
            return ch
        ch[arg[0]] = arg[1]


def select_pivots(risk, count: int):
    """The count units of largest risk (ties: lower index first)."""
    risk = np.asarray(risk, np.float64)
    order = sorted(range(len(risk)), key=lambda u: (-risk[u], u))
    mask = np.zeros(len(risk), bool)
    mask[order[:count]] = True
    return mask
