"""Calibration pipeline of the setup step, on libstepq's host functions:
row-impact factors -> candidate distortions with the dual-axis codec ->
lifetime weights -> FP16 pivots -> bit allocation (Section 3.2, Section 4.3,
Appendices A.3, C.1, C.2).  Argument marshalling only: every step's
arithmetic is a libstepq call.  Produces the precision map (widths 2/4/8, 16 for
pivots) and the row-impact factors a pool is created and refit with."""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from . import stepq


@dataclass
class Calibration:
    row_bits: np.ndarray        # uint8 [H][d_k]: 2, 4, 8 or 16 (pivot)
    row_weight: np.ndarray      # float32 [H][d_k]
    ell: np.ndarray             # mean log retention per unit
    lifetime: np.ndarray        # L_u per unit
    distortion: np.ndarray      # d_u(b) per unit and candidate (16 last if pivots were asked for)


def calibrate(q, k, beta, gates, states, budget: float, cand_bits=(2, 4, 8), unit: str = "row",
              n_pivots: int = 0, horizon: int = 1024, method: str | None = None, gamma: float = 0.25,
              n_threads: int = 0) -> Calibration:
    """q, k [T][H][d_k], beta [T][H], gates [T][H] (GDN) or [T][H][d_k] (KDA):
    calibration activations; states [C][H][d_k][d_v]: sampled reference
    states.  unit "row" (key rows, KDA) or "head" (Qwen); method defaults to
    the Lagrangian for rows and the DP for heads (Appendix C.2).  Pivots are
    the n_pivots units of largest L_u (d_u(b_max) - d_u(16)), chosen first;
    the remaining units are allocated under the budget (pivot bits are
    accounted separately, Table C1)."""
    C, H, dk, dv = np.asarray(states).shape
    w, _ = stepq.stepq_setup_row_impact(q, k, beta, gates, gamma)
    ell = stepq.stepq_setup_mean_log_retention(gates, dk, unit)
    L = stepq.stepq_setup_lifetime_weights(ell, horizon)
    cands = list(cand_bits) + ([16] if n_pivots > 0 else [])
    d = stepq.stepq_setup_distortion(states, cands, unit, row_weight=w, n_threads=n_threads)
    U = d.shape[0]
    piv = np.zeros(U, bool)
    if n_pivots > 0:
        ib = int(np.argmax(cand_bits))
        piv = stepq.stepq_setup_select_pivots(stepq.stepq_setup_pivot_risk(L, d, ib, d.shape[1] - 1), n_pivots)
        # with the pivots fixed, the integer candidates are calibrated again
        # without them in the shared column fit
        pmask = piv.reshape(H, dk) if unit == "row" else np.repeat(piv[:, None], dk, axis=1)
        d_int = stepq.stepq_setup_distortion(states, list(cand_bits), unit, row_weight=w, pivots=pmask,
                                             n_threads=n_threads)
    else:
        d_int = d
    idx = np.nonzero(~piv)[0]
    n_u = np.full(len(idx), dv if unit == "row" else dk * dv, np.int32)
    m = method or ("lagrangian" if unit == "row" else "dp")
    cost = stepq.stepq_setup_lifetime_costs(L, d_int, len(cand_bits))
    choice = stepq.stepq_setup_allocate(cost[idx], n_u, cand_bits, budget, m)
    widths = np.full(U, 16, np.uint8)
    widths[idx] = np.asarray(cand_bits, np.uint8)[choice]
    bits = widths.reshape(H, dk) if unit == "row" else np.repeat(widths[:, None], dk, axis=1)
    return Calibration(bits.astype(np.uint8), w, ell, L, d)
