"""Test-side helpers: drive the oracle and the HIP path on the same seeded
draws and compare them to the tolerances of the decode step.

Protocol (lockstep, re-anchored from the oracle): the oracle runs its own
trajectory from its own quantization of the initial state.  Before each
step the checked GPU slots are overwritten (stepq_pool_import) with the
oracle's previous codes and scales, the GPU step runs at full size, and its
exported codes and outputs for those slots are compared with the oracle's
next step.  Every oracle input comes from the workload draws or from the
oracle itself, never from the GPU.

Tolerances:
  codes   bit-exact, except that at most 1e-4 of the entries compared over a
          run may differ by exactly one level, and only where the oracle's
          unrounded value lies within TIE_WINDOW of a rounding boundary (a tie
          that fp32 and fp64 may break differently); a single step may not
          exceed 1e-3 (STEP_MISMATCH_FRAC);
  outputs |o_gpu - o_oracle| <= 1e-5 + 1e-3 |o_oracle| element-wise.
"""
from __future__ import annotations

import numpy as np
import torch

import oracle
from paper_2609_38169_amd import workloads as W

CODE_MISMATCH_FRAC = 1e-4
STEP_MISMATCH_FRAC = 1e-3
TIE_WINDOW = 2e-3          # code units; fp32 error of the code-space update is ~1e-5
O_ABS, O_REL = 1e-5, 1e-3
# Refitted scales (fp32 sums on the GPU vs fp64): a scale is an fp32 value
# formed from O(d) terms, so 1e-5 relative is ~100 ulp of headroom.  A
# column factor may also come from another, equally valid, rounding of fixed
# codes that sit within TIE_WINDOW of a rounding boundary: the oracle bounds
# the factor over all such roundings (c_range) and the GPU's must lie inside.
SCALE_REL = 1e-5
# Pivot rows hold X rounded to binary16.  X carries the fp32 error of the
# update (~1e-7 of its terms), and binary16 spacing is only 2^-11 relative,
# so fp32 and fp64 land on different sides of a binary16 rounding boundary
# about 2e-4 of the time (codes, with spacing 1 on values up to 127, see
# ties ~20x less often).  Each pivot value is checked to be a correct
# rounding of X within the fp32 error; at most PIVOT_MISMATCH_FRAC may
# differ from the oracle's.
PIVOT_MISMATCH_FRAC = 2e-3


def bits_for(w: W.Workload, layer: int = 0) -> np.ndarray:
    """Bit map from the oracle's own setup (lifetime ranking) or the draw."""
    if w.bits == "lifetime48":
        return oracle.lifetime_bitmap(W.calibration_gates(w, layer).numpy(), w.d_k, budget=6.0)
    return W.bit_map_draw(w, layer).numpy()


def oracle_inputs(w: W.Workload, inp: dict, rows: np.ndarray):
    """Per-tile fp64 activations for batch rows ``rows`` (all heads), exact
    widenings of the stored dtype; q/k expanded over grouped heads."""
    g = w.n_v_heads // w.n_qk_heads
    hq = np.arange(w.n_v_heads) // g
    rows_t = torch.as_tensor(rows, dtype=torch.long, device=inp["q"].device)
    q = inp["q"].index_select(0, rows_t).double().cpu().numpy()[:, hq, :]
    k = inp["k"].index_select(0, rows_t).double().cpu().numpy()[:, hq, :]
    v = inp["v"].index_select(0, rows_t).double().cpu().numpy()
    a = inp["alpha"].index_select(0, rows_t).double().cpu().numpy()
    b = inp["beta"].index_select(0, rows_t).double().cpu().numpy()
    n = len(rows) * w.n_v_heads
    # alpha [B][Hv] (GDN) or channel-wise gates [B][Hv][d_k] (KDA)
    return (q.reshape(n, w.d_k), k.reshape(n, w.d_k), v.reshape(n, w.d_v), a.reshape((n,) + a.shape[2:]),
            b.reshape(n))


FP32_EPS = 2.0 ** -24


def fp32_step_bounds(codes, r, c, bits, q, k, v, alpha, beta, levels: int = 0):
    """Forward error bounds of an fp32 evaluation of the frozen-scale step
    (any summation order, dot products of length d_k), from the oracle's
    own inputs: per code, in code units, and per output.  Used where the
    inputs' dynamic range makes the fixed tie window too narrow: with
    u_j = sum_i g_i k_i S_ij (g = alpha, or the channel gate d),
    delta_j = v_j - u_j and X_ij = g_i S_ij + beta k_i delta_j,
        |d delta_j| <= gam sum_i |g_i k_i S_ij| + 4 eps |v_j|
        |d y_ij|    <= (4 eps (|g_i S_ij| + |beta k_i delta_j|) + |beta k_i| |d delta_j|) / (r_i c_j nu_i)
        |d o_j|     <= gam sum_i |g_i q_i S_ij| + |beta| (|kappa| |d delta_j| + gam sum_i |q_i k_i| |delta_j|)
                       + 4 eps |o_j|
    with gam = (d_k + 8) eps and nu_i the level step of row i."""
    n, dk, dv = codes.shape
    S = oracle.dequant(codes, r, c, bits, levels=levels)
    a = np.asarray(alpha, np.float64)
    g = np.broadcast_to(a.reshape(n, -1), (n, dk)) if a.ndim > 1 else np.broadcast_to(a.reshape(n, 1), (n, dk))
    bw = np.broadcast_to(bits, (n, dk)).astype(np.float64)
    nu = np.exp2(8.0 - bw) if levels else 1.0 / (np.exp2(bw - 1) - 1)
    beta = np.asarray(beta, np.float64).reshape(n, 1)
    eps, gam = FP32_EPS, (dk + 8) * FP32_EPS
    gks = (g * k)[:, :, None] * S
    u = gks.sum(axis=1)
    delta = v - u
    d_delta = gam * np.abs(gks).sum(axis=1) + 4 * eps * np.abs(v)
    X = g[:, :, None] * S + (beta * k)[:, :, None] * delta[:, None, :]
    scale = 1.0 / (np.asarray(r, np.float64)[:, :, None] * np.asarray(c, np.float64)[:, None, :] * nu[:, :, None])
    dy = (4 * eps * (np.abs(g[:, :, None] * S) + np.abs((beta * k)[:, :, None] * delta[:, None, :]))
          + np.abs(beta * k)[:, :, None] * d_delta[:, None, :]) * scale
    kappa = (q * k).sum(axis=1, keepdims=True)
    o = (X * q[:, :, None]).sum(axis=1)
    do = (gam * np.abs((g * q)[:, :, None] * S).sum(axis=1)
          + np.abs(beta) * (np.abs(kappa) * d_delta + gam * np.abs(q * k).sum(axis=1, keepdims=True) * np.abs(delta))
          + 4 * eps * np.abs(o))
    return dy, do


def compare_codes(gpu: np.ndarray, orc: np.ndarray, y: np.ndarray, what: str = "codes",
                  frac: float = CODE_MISMATCH_FRAC, window=TIE_WINDOW, total: int | None = None):
    """Apply the code tolerance to one comparison (at most ``frac`` of the
    entries mismatched, each within ``window`` of a rounding tie: a scalar
    or a per-code array); returns the number of tie mismatches.  ``total``:
    the number of entries the fraction applies to, when the arrays passed
    are the part of a larger comparison that holds every mismatch."""
    diff = gpu.astype(np.int16) - orc.astype(np.int16)
    bad = np.nonzero(diff)
    n_bad = bad[0].size
    if n_bad == 0:
        return 0
    assert np.all(np.abs(diff[bad]) == 1), f"{what}: a code differs by more than one level"
    fpart = np.abs(y[bad]) - np.floor(np.abs(y[bad]))
    win = np.broadcast_to(window, y.shape)[bad]
    near_tie = np.abs(fpart - 0.5) <= win
    assert np.all(near_tie), (f"{what}: {int((~near_tie).sum())} mismatches away from a rounding tie, e.g. "
                              f"y={y[bad][~near_tie][:4]}")
    total = gpu.size if total is None else total
    assert n_bad <= frac * total, f"{what}: {n_bad} of {total} codes differ"
    return n_bad


def compare_refit(g_codes, g_r, g_c, o_codes, o_r, o_c, y, c_range, bits, what: str = "refit",
                  frac: float = CODE_MISMATCH_FRAC):
    """Tolerances of the refitting step, tile arrays [n][dk][dv], [n][dk],
    [n][dv].  Returns (codes that differ from the oracle's, columns whose
    factor differs from the oracle's by more than SCALE_REL); the first is
    held to CODE_MISMATCH_FRAC over a run by the caller.

    r' within SCALE_REL.  c' within SCALE_REL of the oracle's range over the
    near-tie roundings of its fixed codes.  Codes: the oracle's state X
    quantized with the GPU's (admissible) scales, i.e. y scaled by
    (r_orc / r_gpu)(c_orc / c_gpu); the GPU's codes must equal its rounding,
    except by one level within TIE_WINDOW of a rounding boundary, for at most
    ``frac`` of the entries.  (Where the GPU took the other rounding of a tie
    in the fixed codes, a whole column's factor moves and many of its codes
    may then differ from the oracle's own, each correctly rounded.)"""
    g_r, g_c = g_r.astype(np.float64), g_c.astype(np.float64)
    o_r, o_c = o_r.astype(np.float64), o_c.astype(np.float64)
    dr = np.abs(g_r - o_r) / o_r
    assert np.all(dr <= SCALE_REL), f"{what}: row scale off by {dr.max():.3g} relative"
    lo, hi = c_range
    inside = (g_c >= lo * (1 - SCALE_REL)) & (g_c <= hi * (1 + SCALE_REL))
    assert np.all(inside), (f"{what}: {int((~inside).sum())} column scales outside the admissible range, e.g. "
                            f"{g_c[~inside][:3]} vs [{lo[~inside][:3]}, {hi[~inside][:3]}]")
    dc = np.abs(g_c - o_c) / o_c
    qb = (2.0 ** (bits.astype(np.int64) - 1) - 1)[:, :, None]
    ys = y * (o_r / g_r)[:, :, None] * (o_c / g_c)[:, None, :]
    expect = np.clip(np.rint(ys), -qb, qb).astype(np.int16)
    expect[np.broadcast_to((bits == 16)[:, :, None], expect.shape)] = 0     # pivot rows carry no codes
    diff = g_codes.astype(np.int16) - expect
    bad = np.nonzero(diff)
    n_bad = bad[0].size
    if n_bad:
        assert np.all(np.abs(diff[bad]) == 1), (f"{what}: a code differs by more than one level from the rounding "
                                                f"under the GPU scales, e.g. y={ys[bad][:3]} got {g_codes[bad][:3]}")
        yb = np.abs(ys[bad])
        fpart = yb - np.floor(yb)
        ok = np.abs(fpart - 0.5) <= TIE_WINDOW
        assert np.all(ok), (f"{what}: {int((~ok).sum())} code mismatches not at a rounding tie, e.g. "
                            f"y={ys[bad][~ok][:4]}")
        assert n_bad <= frac * g_codes.size, f"{what}: {n_bad} of {g_codes.size} codes differ"
    return int(np.count_nonzero(g_codes != o_codes)), int((dc > SCALE_REL).sum())


def _half_ulp(x):
    """Spacing of binary16 values around |x| (subnormal spacing 2^-24)."""
    a = np.abs(x)
    e = np.floor(np.log2(np.where(a > 0, a, 1.0)))
    return np.exp2(np.maximum(e - 10, -24))


def compare_pivots(g_pv, o_pv, X, mask, what: str = "pivots", frac: float = PIVOT_MISMATCH_FRAC):
    """Pivot rows (mask [n][dk]): the GPU's binary16 value must be a correct
    rounding of the oracle's X up to the error of X in fp32 arithmetic (1% of
    half a binary16 spacing, or 1e-6 of the row's largest |X| for values near
    zero, where X is a difference of much larger terms), so it can differ from
    the oracle's own rounding only at a rounding tie; at most one value plus
    ``frac`` of them may differ (a single comparison holds only a few
    thousand pivot values).  Returns the number that differ."""
    sel = np.broadcast_to(mask[:, :, None], g_pv.shape)
    g = g_pv[sel].view(np.float16).astype(np.float64)
    x = X[sel]
    row_mag = np.broadcast_to(np.abs(X).max(axis=2, keepdims=True), X.shape)[sel]
    allow = 0.5 * _half_ulp(x) * 1.01 + 1e-6 * row_mag
    assert np.all(np.abs(g - x) <= allow), \
        f"{what}: a pivot value is not a binary16 rounding of X (max err {np.max(np.abs(g - x) / _half_ulp(x)):.3f} ulp)"
    n_bad = int(np.count_nonzero(g_pv[sel] != o_pv[sel]))
    assert n_bad <= 1 + frac * g.size, f"{what}: {n_bad} of {g.size} pivot values differ"
    return n_bad


def compare_out(gpu: np.ndarray, orc: np.ndarray, what: str = "o", bound=None):
    """|o_gpu - o_oracle| within O_ABS + O_REL |o_oracle|, or within
    ``bound`` (per output) where that is larger."""
    err = np.abs(gpu.astype(np.float64) - orc)
    lim = O_ABS + O_REL * np.abs(orc)
    if bound is not None:
        lim = np.maximum(lim, bound)
    worst = np.argmax(err - lim)
    assert np.all(err <= lim), (f"{what}: |diff| {err.flat[worst]:.3g} > {lim.flat[worst]:.3g} "
                                f"(oracle {orc.flat[worst]:.6g}); {int((err > lim).sum())} entries out")


class Lockstep:
    """One workload layer: a GPU pool plus the oracle's trajectory on
    ``check_rows`` (batch rows whose slots are compared each step).

    Every code compared is counted once in ``compared``; ``mismatches``
    counts the codes that differ from the oracle's (ties).  ``finish``
    applies the run-level limits.  Frozen steps without pivot rows or fp32
    bounds take a fast path: the oracle's unrounded values are formed only
    for the tiles that hold a mismatch, which keeps a check of every tile of
    a 16,384-tile launch to about a second per step."""

    def __init__(self, w: W.Workload, pool, slots: torch.Tensor, bits: np.ndarray, check_rows: np.ndarray,
                 S0_check: np.ndarray, layer: int = 0, refit=False, row_weight=None, levels: int = 0,
                 fp32_bounds: bool = False):
        self.w, self.pool, self.slots, self.bits, self.layer = w, pool, slots, bits, layer
        self.fp32_bounds = fp32_bounds      # o limit (and the frozen steps' tie window) from fp32_step_bounds
        self.refit = refit
        self.lv = dict(levels=levels)
        self.tie_cols = 0
        self.rows = np.asarray(check_rows)
        n = len(self.rows) * w.n_v_heads
        self.tile_bits = np.broadcast_to(bits[None], (len(self.rows),) + bits.shape).reshape(n, w.d_k)
        S = S0_check.reshape(n, w.d_k, w.d_v)
        self.pivots = bool(np.any(bits == 16))
        self.r, self.c = oracle.fit_absmax(S, bits=self.tile_bits, **self.lv)
        q = oracle.quantize(S.astype(np.float64), self.r, self.c, self.tile_bits, **self.lv)
        self.codes, self.pv = (q[0], q[1]) if self.pivots else (q, None)
        self.piv_mismatches = 0
        self.piv_compared = 0
        dev = pool.device
        self.ids = slots.index_select(0, torch.as_tensor(self.rows, dtype=torch.long, device=slots.device)).to(dev)
        self.n_tiles = n
        self.row_w = None if row_weight is None else np.broadcast_to(
            np.asarray(row_weight, np.float64)[None], (len(self.rows),) + bits.shape).reshape(n, w.d_k)
        self.mismatches = 0
        self.compared = 0
        self.steps = 0

    @property
    def saturated(self) -> float:
        """Fraction of the oracle's current integer codes at +-q_b."""
        qb = (2 ** (np.minimum(self.tile_bits, 8).astype(np.int32) - 1) - 1).astype(np.int8)[:, :, None]
        ints = np.broadcast_to((self.tile_bits != 16)[:, :, None], self.codes.shape)
        sat = (np.abs(self.codes) == qb) & ints
        return float(sat.sum()) / max(1, int(ints.sum()))

    def shaped(self, a, tail):
        return a.reshape((len(self.rows), self.w.n_v_heads) + tail)

    def anchor(self):
        """Write the oracle's current state into the checked GPU slots."""
        w, dev = self.w, self.pool.device
        self.pool.import_(self.ids,
                          torch.from_numpy(np.ascontiguousarray(self.shaped(self.codes, (w.d_k, w.d_v)))).to(dev),
                          torch.from_numpy(np.ascontiguousarray(self.shaped(self.r, (w.d_k,)))).to(dev),
                          torch.from_numpy(np.ascontiguousarray(self.shaped(self.c, (w.d_v,)))).to(dev))
        if self.pivots:
            pv = np.ascontiguousarray(self.shaped(self.pv, (w.d_k, w.d_v))).view(np.int16)
            self.pool.import_pivots(self.ids, torch.from_numpy(pv).to(dev))

    def export(self):
        w, dev = self.w, self.pool.device
        n = len(self.rows)
        codes = torch.empty((n, w.n_v_heads, w.d_k, w.d_v), dtype=torch.int8, device=dev)
        r = torch.empty((n, w.n_v_heads, w.d_k), dtype=torch.float32, device=dev)
        c = torch.empty((n, w.n_v_heads, w.d_v), dtype=torch.float32, device=dev)
        self.pool.export(self.ids, codes, r, c)
        self.g_pv = None
        if self.pivots:
            pv = torch.empty((n, w.n_v_heads, w.d_k, w.d_v), dtype=torch.int16, device=dev)
            self.pool.export_pivots(self.ids, pv)
            self.g_pv = pv.cpu().numpy().view(np.uint16).reshape(self.n_tiles, w.d_k, w.d_v)
        if codes.is_cuda:
            torch.cuda.synchronize()
        return codes.cpu().numpy().reshape(self.n_tiles, w.d_k, w.d_v), r.cpu().numpy(), c.cpu().numpy()

    def _frozen_fast(self, g_codes, q, k, v, a, b, step):
        """Frozen step, every tile compared; y only where codes differ."""
        new, o = oracle.decode_step(self.codes, self.r, self.c, self.tile_bits, q, k, v, a, b, **self.lv)
        diff_tiles = np.nonzero(np.any((g_codes != new).reshape(self.n_tiles, -1), axis=1))[0]
        nb = 0
        if diff_tiles.size:
            t = diff_tiles
            _, _, y = oracle.decode_step(self.codes[t], self.r[t], self.c[t], self.tile_bits[t], q[t], k[t], v[t],
                                         a[t], b[t], want_y=True, **self.lv)
            nb = compare_codes(g_codes[t], new[t], y, f"layer {self.layer} step {step} codes",
                               frac=STEP_MISMATCH_FRAC, total=g_codes.size)
        return new, o, nb

    def check_step(self, inp: dict, o_gpu: torch.Tensor, step: int):
        """Oracle step on its own state, compare with the GPU's result."""
        w = self.w
        q, k, v, a, b = oracle_inputs(w, inp, self.rows)
        g_codes, g_r, g_c = self.export()
        pvk = dict(pv=self.pv) if self.pivots else {}
        pmask = self.tile_bits == 16
        o_bound = dy = None
        if self.fp32_bounds:
            assert not self.pivots, "fp32 step bounds cover integer rows only"
            dy, o_bound = fp32_step_bounds(self.codes, self.r, self.c, self.tile_bits, q, k, v, a, b,
                                           self.lv["levels"])
        if self.refit == "row_absmax":
            res = oracle.decode_step_rowmax(self.codes, self.r, self.c, self.tile_bits, q, k, v, a, b, want_y=True,
                                            **pvk, **self.lv)
            new, rn, cn, o, y = res[:5]
            if self.pivots:
                self.piv_mismatches += compare_pivots(self.g_pv, res[5], y, pmask, f"step {step} pivots")
                self.pv = res[5]
            g_c = g_c.reshape(cn.shape)
            assert np.all(g_c == 1.0), "row-absmax step: column factors must all be 1"
            ones = np.ones(cn.shape, np.float64)
            nb, _ = compare_refit(g_codes, g_r.reshape(rn.shape), g_c, new, rn, cn, y, (ones, ones),
                                  self.tile_bits, f"layer {self.layer} step {step} row absmax",
                                  frac=STEP_MISMATCH_FRAC)
            self.r, self.c = rn, cn
        elif self.refit:
            res = oracle.decode_step_refit(self.codes, self.r, self.c, self.tile_bits, q, k, v, a, b,
                                           w=self.row_w, want=("y", "c_range"), tie_window=TIE_WINDOW, **pvk,
                                           **self.lv)
            new, rn, cn, o, ex = res[:5]
            if self.pivots:
                self.piv_mismatches += compare_pivots(self.g_pv, res[5], ex["y"], pmask, f"step {step} pivots")
                self.pv = res[5]
            nb, tc = compare_refit(g_codes, g_r.reshape(rn.shape), g_c.reshape(cn.shape), new, rn, cn,
                                   ex["y"], ex["c_range"], self.tile_bits, f"layer {self.layer} step {step} refit",
                                   frac=STEP_MISMATCH_FRAC)
            self.tie_cols += tc
            self.r, self.c = rn, cn
        else:
            assert np.array_equal(g_r.reshape(self.r.shape), self.r), "row scales changed"
            assert np.array_equal(g_c.reshape(self.c.shape), self.c), "column scales changed"
            if dy is None and not self.pivots:
                new, o, nb = self._frozen_fast(g_codes, q, k, v, a, b, step)
            else:
                res = oracle.decode_step(self.codes, self.r, self.c, self.tile_bits, q, k, v, a, b, want_y=True,
                                         **pvk, **self.lv)
                new, o, y = res[:3]
                if self.pivots:
                    self.piv_mismatches += compare_pivots(self.g_pv, res[3], y, pmask, f"step {step} pivots")
                    self.pv = res[3]
                win = TIE_WINDOW if dy is None else TIE_WINDOW + dy
                nb = compare_codes(g_codes, new, y, f"layer {self.layer} step {step} codes",
                                   frac=STEP_MISMATCH_FRAC, window=win)
        self.mismatches += nb
        self.compared += g_codes.size
        if self.pivots:
            self.piv_compared += int(np.count_nonzero(pmask)) * w.d_v
        rows_t = torch.as_tensor(self.rows, dtype=torch.long, device=o_gpu.device)
        og = o_gpu.index_select(0, rows_t).cpu().numpy().reshape(self.n_tiles, w.d_v)
        compare_out(og, o, f"layer {self.layer} step {step} o", bound=o_bound)
        self.codes = new
        self.steps += 1

    def finish(self, what: str = ""):
        """Run-level limits: codes that differ from the oracle's at most
        CODE_MISMATCH_FRAC of the codes compared over the run, pivot values at
        most PIVOT_MISMATCH_FRAC (plus one)."""
        assert self.compared > 0, f"{what}: nothing compared"
        assert self.mismatches <= CODE_MISMATCH_FRAC * self.compared, \
            f"{what}: {self.mismatches} of {self.compared} codes differ over the run"
        if self.pivots:
            assert self.piv_mismatches <= PIVOT_MISMATCH_FRAC * self.piv_compared + 1, \
                f"{what}: {self.piv_mismatches} of {self.piv_compared} pivot values differ over the run"
        return self


def lockstep_run(w: W.Workload, steps: int, check_rows, device, layer: int = 0, mutate=None, kda: bool = False,
                 refit=False, row_weight=None, say=print, bits=None, levels: int = 0, state_map=None,
                 fp32_bounds: bool = False, every: int = 16):
    """Full-size decode steps of one workload layer on the GPU, the rows
    ``check_rows`` compared lockstep with the oracle at every step.
    ``state_map`` (optional) transforms the checked slots' initial states
    [rows][Hv][d_k][d_v] before the oracle fits and quantizes them.
    ``fp32_bounds``: judge o (every mode) and, on frozen steps, the codes'
    distance from a rounding tie against the fp32 forward error bounds of
    the step as well as the fixed limits.  A progress line every ``every``
    steps."""
    from paper_2609_38169_amd.pools import build_pool, row_bits
    bits = row_bits(w, layer) if bits is None else bits
    say(f"lockstep {w.name}: building pool ({w.n_slots} slots), checking {len(check_rows)} of {w.batch} requests")
    pool = build_pool(w, layer, device=device, bits=bits, levels=levels)
    if row_weight is not None:
        pool.set_row_weight(row_weight)
    slots = W.active_slots(w).to(device)
    check_slots = W.active_slots(w)[np.asarray(check_rows)]
    S0 = W.initial_state(w, layer, [int(x) for x in check_slots], device=device).cpu().numpy()
    if state_map is not None:
        S0 = np.ascontiguousarray(state_map(S0), dtype=np.float32)
    ls = Lockstep(w, pool, slots, bits, check_rows, S0, layer, refit=refit, row_weight=row_weight, levels=levels,
                  fp32_bounds=fp32_bounds)
    del S0
    o = torch.empty((w.batch, w.n_v_heads, w.d_v), dtype=torch.float32, device=device)
    for t in range(steps):
        inp = W.step_inputs(w, layer, t, device=device)
        if kda:
            inp["alpha"] = W.kda_gates(w, layer, t, device=device)
        if mutate:
            inp = mutate(inp)
        ls.anchor()
        if kda:
            pool.step_kda(slots, inp["q"], inp["k"], inp["v"], inp["alpha"], inp["beta"], o, refit=refit)
        else:
            pool.step(slots, inp["q"], inp["k"], inp["v"], inp["alpha"], inp["beta"], o, refit=refit)
        torch.cuda.synchronize()
        ls.check_step(inp, o, t)
        if every and (t + 1) % every == 0 and t + 1 < steps:
            say(f"lockstep {w.name}: {t + 1} steps ok ({ls.mismatches} code mismatches of {ls.compared})")
    ls.finish(f"lockstep {w.name}")
    mode = {False: "", True: " refit", "row_absmax": " row-absmax"}[refit] + (" N2 levels" if levels else "")
    say(f"lockstep {w.name}{' kda' if kda else ''}{mode}: {steps} steps ok, "
        f"{ls.compared} codes compared, code mismatches {ls.mismatches}, pivot mismatches {ls.piv_mismatches}, "
        f"columns on another tie rounding {ls.tie_cols}, "
        f"saturated {ls.saturated:.3f}")
    return ls
