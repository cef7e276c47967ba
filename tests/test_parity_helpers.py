"""The comparison rules of the GPU parity tests, exercised on the CPU with
planted differences (the rules themselves must accept what the tolerances
allow and reject everything else)."""
import numpy as np
import pytest
import torch

import _parity as PT
import oracle


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


def _fp32_step(codes, r, c, bits, q, k, v, alpha, beta, split: bool):
    """The frozen step's code-space form evaluated in fp32 (the decode
    kernel's arithmetic): weights k r 2^(b-8)/q_b, optionally rounded to the
    binary16 hi + lo pair under a power-of-two prescale per tile; y in code
    units and o."""
    f32 = np.float32
    n, dk, dv = codes.shape
    bw = bits.astype(np.int64)
    qb = np.exp2(bw - 1) - 1
    U = (codes.astype(np.float64) * np.exp2(8 - bw)[:, :, None]).astype(f32)
    fq = (np.exp2(bw - 8) / qb).astype(f32)
    kt = (k.astype(f32) * (r * fq)).astype(f32)
    qt = (q.astype(f32) * (r * fq)).astype(f32)

    def matvec(wt):
        if split:
            e = np.clip(15 - np.frexp(np.abs(wt).max(axis=1))[1], -126, 126)
            ws = (wt * np.exp2(e)[:, None]).astype(f32)
            hi = ws.astype(np.float16)
            lo = (ws - hi.astype(f32)).astype(np.float16)
            s = np.zeros((n, dv), f32)
            for i in range(dk):
                s = (s + (hi[:, i].astype(f32)[:, None] * U[:, i, :]).astype(f32)
                     + (lo[:, i].astype(f32)[:, None] * U[:, i, :]).astype(f32)).astype(f32)
            return (s * np.exp2(-e)[:, None]).astype(f32)
        s = np.zeros((n, dv), f32)
        for i in range(dk):
            s = (s + wt[:, i, None] * U[:, i, :]).astype(f32)
        return s

    al = alpha.astype(f32)[:, None]
    b32 = beta.astype(f32)[:, None]
    cu = (c * matvec(kt)).astype(f32)
    cp = (c * matvec(qt)).astype(f32)
    delta = (v.astype(f32) - al * cu).astype(f32)
    kappa = (q.astype(f32) * k.astype(f32)).sum(axis=1, dtype=f32)[:, None]
    o = (al * cp + b32 * kappa * delta).astype(f32)
    ai = (b32 * k.astype(f32) * qb.astype(f32) * (f32(1) / r)).astype(f32)
    bcol = (delta * (f32(1) / c)).astype(f32)
    y = (al[:, :, None] * np.exp2(bw - 8).astype(f32)[:, :, None] * U + ai[:, :, None] * bcol[:, None, :]).astype(f32)
    return y, o


@pytest.mark.parametrize("spread", [(0, 0, 0, 0), (-4, 4, -16, 16)])
def test_fp32_step_bounds_cover_fp32_evaluations(spread):
    """The per-code and per-output bounds used for wide-range GPU cases hold
    for fp32 evaluations of the step (the code-space form with fp32 weights,
    and with the binary16 hi + lo weight split), on ordinary tiles and on
    tiles whose weights span ~40 binades."""
    s_lo, s_hi, k_lo, k_hi = spread
    rng = np.random.default_rng(11)
    n, dk, dv = 8, 128, 128
    bits = rng.choice(np.array([4, 8], np.uint8), size=(n, dk))
    S = rng.normal(0.0, 0.05, (n, dk, dv)) * np.exp2(rng.integers(s_lo, s_hi + 1, (n, dk, 1)))
    r, c = oracle.fit_absmax(S.astype(np.float32), bits=bits)
    codes = oracle.quantize(S, r, c, bits)
    unit = lambda x: x / np.linalg.norm(x, axis=1, keepdims=True)
    q = unit(rng.normal(size=(n, dk))).astype(np.float32).astype(np.float64)
    k = (unit(rng.normal(size=(n, dk))) * np.exp2(rng.integers(k_lo, k_hi + 1, (n, dk)))).astype(np.float32)
    k = k.astype(np.float64)
    v = rng.normal(size=(n, dv)).astype(np.float32).astype(np.float64)
    alpha = (1.0 - rng.uniform(0, 0.05, n)).astype(np.float32).astype(np.float64)
    beta = rng.uniform(0.1, 0.9, n).astype(np.float32).astype(np.float64)
    _, o64, y64 = oracle.decode_step(codes, r, c, bits, q, k, v, alpha, beta, want_y=True)
    dy, do = PT.fp32_step_bounds(codes, r, c, bits, q, k, v, alpha, beta)
    qb = (np.exp2(bits.astype(np.int64) - 1) - 1)[:, :, None]
    live = np.abs(y64) < qb + 0.5          # clamped codes do not depend on the error
    if spread == (0, 0, 0, 0):
        # on ordinary tiles the bound is tighter than the fixed tie window
        assert np.quantile(dy[live], 0.999) < PT.TIE_WINDOW
    else:
        # and where fp32 cannot resolve a code it widens the window for few codes only
        assert np.mean(dy[live] > 0.05) < 0.01
    for split in (False, True):
        y, o = _fp32_step(codes, r, c, bits, q, k, v, alpha, beta, split)
        assert np.all(np.abs(y.astype(np.float64) - y64)[live] <= dy[live]), split
        assert np.all(np.abs(o.astype(np.float64) - o64) <= do), split


# --- run-level counting of the lockstep (Lockstep.check_step / finish) ------

class _HostPool:
    """Stand-in for a pool in host memory: ``import_`` records what the
    lockstep anchors; ``export`` returns the result the test planted."""

    device = torch.device("cpu")

    def __init__(self):
        self.result = None

    def import_(self, ids, codes, r, c):
        self.anchored = (codes.numpy().copy(), r.numpy().copy(), c.numpy().copy())

    def export(self, ids, codes, r, c):
        g_codes, g_r, g_c = self.result
        codes.copy_(torch.from_numpy(g_codes.reshape(codes.shape)))
        r.copy_(torch.from_numpy(np.ascontiguousarray(g_r, np.float32).reshape(r.shape)))
        c.copy_(torch.from_numpy(np.ascontiguousarray(g_c, np.float32).reshape(c.shape)))


def _flip_ties(codes, y, bits, n_flip, rng):
    """The other rounding of ``n_flip`` codes whose unrounded value lies
    within the tie window (and away from the clip)."""
    qb = (2.0 ** (bits.astype(np.int64) - 1) - 1)[:, :, None]
    fpart = np.abs(y) - np.floor(np.abs(y))
    cand = np.argwhere((np.abs(fpart - 0.5) <= PT.TIE_WINDOW) & (np.abs(y) < qb - 1))
    assert len(cand) >= n_flip, "too few near-tie codes in the draw"
    g = codes.copy()
    for t, i, j in cand[rng.choice(len(cand), n_flip, replace=False)]:
        lo = np.floor(y[t, i, j])
        g[t, i, j] = int(lo + 1) if g[t, i, j] == lo else int(lo)
    return g


def _host_lockstep_run(mode, flips_per_step, steps=32):
    """The tiny workload driven through Lockstep with the oracle's own step
    standing in for the GPU's, plus planted tie flips."""
    from paper_2609_38169_amd import workloads as W
    from paper_2609_38169_amd.pools import row_bits
    w = W.workload(0)
    bits = row_bits(w)
    rows = np.arange(w.batch)
    S0 = W.initial_state(w, 0, [int(s) for s in W.active_slots(w)[rows]]).numpy()
    pool = _HostPool()
    ls = PT.Lockstep(w, pool, W.active_slots(w), bits, rows, S0, refit=mode)
    rng = np.random.default_rng(5)
    for t in range(steps):
        inp = W.step_inputs(w, 0, t)
        ls.anchor()
        q, k, v, a, b = PT.oracle_inputs(w, inp, rows)
        if mode == "refit":
            new, rn, cn, o, ex = oracle.decode_step_refit(ls.codes, ls.r, ls.c, ls.tile_bits, q, k, v, a, b,
                                                          want=("y",))
            y = ex["y"]
        elif mode == "row_absmax":
            new, rn, cn, o, y = oracle.decode_step_rowmax(ls.codes, ls.r, ls.c, ls.tile_bits, q, k, v, a, b,
                                                          want_y=True)
        else:
            new, o, y = oracle.decode_step(ls.codes, ls.r, ls.c, ls.tile_bits, q, k, v, a, b, want_y=True)
            rn, cn = ls.r, ls.c
        pool.result = (_flip_ties(new, y, ls.tile_bits, flips_per_step, rng), rn, cn)
        o_gpu = torch.from_numpy(o.astype(np.float32).reshape(w.batch, w.n_v_heads, w.d_v))
        ls.check_step(inp, o_gpu, t)
    return ls


@pytest.mark.parametrize("mode", ["refit", "row_absmax", False])
def test_lockstep_counts_each_code_once(mode):
    """1.5e-4 of the codes compared over a run differ at ties: each step is
    within its 1e-3 limit, the run is beyond the 1e-4 limit and must fail
    (each code counted once); 0.6e-4 passes."""
    steps, per_tile = 32, 64 * 64
    ls = _host_lockstep_run(mode, flips_per_step=3, steps=steps)
    assert ls.compared == steps * 4 * per_tile
    assert ls.mismatches == 3 * steps and ls.mismatches > 1.4e-4 * ls.compared
    with pytest.raises(AssertionError, match="differ over the run"):
        ls.finish()
    ls = _host_lockstep_run(mode, flips_per_step=1, steps=steps)
    assert ls.mismatches == steps and ls.mismatches < 0.7e-4 * ls.compared
    ls.finish()


def test_lockstep_fast_path_rejects_non_tie_mismatch():
    """The frozen fast path forms the oracle's unrounded values only for
    tiles with a mismatch; a mismatch away from a tie still fails."""
    from paper_2609_38169_amd import workloads as W
    from paper_2609_38169_amd.pools import row_bits
    w = W.workload(0)
    bits = row_bits(w)
    rows = np.arange(w.batch)
    S0 = W.initial_state(w, 0, [int(s) for s in W.active_slots(w)[rows]]).numpy()
    pool = _HostPool()
    ls = PT.Lockstep(w, pool, W.active_slots(w), bits, rows, S0)
    inp = W.step_inputs(w, 0, 0)
    ls.anchor()
    q, k, v, a, b = PT.oracle_inputs(w, inp, rows)
    new, o, y = oracle.decode_step(ls.codes, ls.r, ls.c, ls.tile_bits, q, k, v, a, b, want_y=True)
    fpart = np.abs(y) - np.floor(np.abs(y))
    t, i, j = np.argwhere((np.abs(fpart - 0.5) > 0.3) & (np.abs(y) < 3))[0]
    g = new.copy()
    g[t, i, j] += 1
    pool.result = (g, ls.r, ls.c)
    with pytest.raises(AssertionError, match="away from a rounding tie"):
        ls.check_step(inp, torch.from_numpy(o.astype(np.float32).reshape(w.batch, w.n_v_heads, w.d_v)), 0)
