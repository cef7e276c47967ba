"""GPU parity with FP16 pivot rows (width 16 in the precision map): layout
round trips, boundary pack, reconstruction, and the decode step in all three
scale modes (frozen, dual-axis refit, row-absmax baseline), GDN and KDA,
against the fp64 oracle through the C ABI."""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_38169_amd import stepq, workloads as W
from paper_2609_38169_amd.pools import row_bits
import _parity as PT

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda", 0)


def _say(*a):
    print(*a, flush=True)


def _cases():
    rng = np.random.default_rng(11)
    cases = []
    for (Hv, Hqk, dk, dv, n_slots, npiv) in [(3, 1, 37, 64, 5, 3), (2, 2, 96, 128, 4, 5), (4, 2, 128, 128, 3, 2),
                                             (2, 1, 128, 128, 2, 32), (1, 1, 1, 64, 2, 1)]:
        bits = rng.choice([2, 4, 8], size=(Hv, dk)).astype(np.uint8)
        for h in range(Hv):
            if h % 2 == 0 or Hv == 1:
                bits[h, rng.choice(dk, size=min(npiv, dk), replace=False)] = 16
        cases.append((Hv, Hqk, dk, dv, n_slots, bits))
    # whole FP16 heads (the paper's Qwen pivots are entire heads): every other
    # head of random widths, then one FP16 head beside 64@8 + 64@4 heads
    bits = rng.choice([2, 4, 8], size=(4, 128)).astype(np.uint8)
    bits[0::2] = 16
    cases.append((4, 2, 128, 128, 3, bits))
    bits = np.stack([rng.permutation(np.repeat(np.array([8, 4], np.uint8), 64)) for _ in range(4)])
    bits[1] = 16
    cases.append((4, 4, 128, 128, 3, bits))

    # heads of a uniform mix with some rows turned into FP16 pivots: stored
    # padded to the mix and run by its compiled body (with the pivot rows)
    def mix(counts, n_heads):
        row = np.concatenate([np.full(n, b, np.uint8) for b, n in counts])
        return np.stack([rng.permutation(row) for _ in range(n_heads)])

    def pivots(bits, heads, n):
        for h, k in zip(heads, n):
            bits[h, rng.choice(128, size=k, replace=False)] = 16
        return bits

    six, four = [(8, 64), (4, 64)], [(8, 32), (4, 32), (2, 64)]
    # 7: every head a padded pivot head of 64@8 + 64@4 (1 to 8 pivots)
    cases.append((4, 2, 128, 128, 3, pivots(mix(six, 4), range(4), [1, 3, 5, 8])))
    # 8: 32@8 + 32@4 + 64@2 heads, two of them with pivots (uniform and pivot heads in one launch)
    cases.append((4, 4, 128, 128, 3, pivots(mix(four, 4), [1, 2], [2, 7])))
    # 9: all-8, all-4 and all-2 heads with pivots (one launch per class)
    b9 = np.concatenate([mix([(8, 128)], 2), mix([(4, 128)], 2), mix([(2, 128)], 2)])
    cases.append((6, 3, 128, 128, 3, pivots(b9, range(6), [2, 1, 4, 8, 3, 6])))
    # 10: 64@8 + 64@4 heads, a pivot one, a compact generic one (random widths,
    # 2 pivots), and one with 10 pivots (padded, on the generic body)
    b10 = mix(six, 4)
    b10[2] = rng.choice([2, 4, 8], size=128).astype(np.uint8)
    cases.append((4, 2, 128, 128, 3, pivots(b10, [1, 2, 3], [4, 2, 10])))
    # 11: 64@8 + 64@4 heads, a pivot one and a whole FP16 head
    b11 = pivots(mix(six, 4), [2], [6])
    b11[3] = 16
    cases.append((4, 4, 128, 128, 3, b11))
    return cases


N_CASES = 12


def _state(case, seed):
    Hv, Hqk, dk, dv, n_slots, bits = _cases()[case]
    rng = np.random.default_rng(seed)
    S = (rng.standard_normal((n_slots, Hv, dk, dv)) * 0.05).astype(np.float32)
    tb = np.broadcast_to(bits[None], (n_slots,) + bits.shape).reshape(-1, dk)
    r, c = oracle.fit_absmax(S.reshape(-1, dk, dv), bits=tb)
    codes, pv = oracle.quantize(S.reshape(-1, dk, dv).astype(np.float64), r, c, tb)
    return rng, S, tb, r, c, codes, pv


def _pool_with(case, codes, pv, r, c):
    Hv, Hqk, dk, dv, n_slots, bits = _cases()[case]
    pool = stepq.Pool(n_slots, Hv, Hqk, dk, dv, bits, device=DEV)
    ids = torch.arange(n_slots, dtype=torch.int32, device=DEV)
    pool.import_(ids, torch.from_numpy(codes.reshape(n_slots, Hv, dk, dv)).to(DEV),
                 torch.from_numpy(r.reshape(n_slots, Hv, dk)).to(DEV),
                 torch.from_numpy(c.reshape(n_slots, Hv, dv)).to(DEV))
    pool.import_pivots(ids, torch.from_numpy(pv.reshape(n_slots, Hv, dk, dv).view(np.int16)).to(DEV))
    return pool, ids


@pytest.mark.parametrize("case", range(N_CASES))
def test_pivot_import_export_and_image(case):
    Hv, Hqk, dk, dv, n_slots, bits = _cases()[case]
    _say(f"pivot layout case {case}: Hv={Hv} dk={dk} dv={dv} pivots/head={list((bits == 16).sum(1))}")
    _, S, tb, r, c, codes, pv = _state(case, 500 + case)
    pool, ids = _pool_with(case, codes, pv, r, c)
    img = pool.memory.cpu().numpy()
    shp = (n_slots, Hv, dk, dv)
    assert np.array_equal(img, oracle.pack_pool(codes.reshape(shp), r.reshape(n_slots, Hv, dk),
                                                c.reshape(n_slots, Hv, dv), bits, pv=pv.reshape(shp)))
    oc = torch.empty(shp, dtype=torch.int8, device=DEV)
    opv = torch.empty(shp, dtype=torch.int16, device=DEV)
    pool.export(ids, oc, torch.empty((n_slots, Hv, dk), device=DEV), torch.empty((n_slots, Hv, dv), device=DEV))
    pool.export_pivots(ids, opv)
    deq = torch.empty(shp, dtype=torch.float32, device=DEV)
    pool.dequant(ids, deq)
    torch.cuda.synchronize()
    assert np.array_equal(oc.cpu().numpy().reshape(codes.shape), codes)
    assert np.array_equal(opv.cpu().numpy().view(np.uint16).reshape(pv.shape), pv)
    piv = tb == 16
    d = deq.cpu().numpy().reshape(codes.shape)
    assert np.array_equal(d[piv], oracle.half_to_double(pv)[piv].astype(np.float32))


@pytest.mark.parametrize("case", [0, 2])
def test_pivot_boundary_pack(case):
    """stepq_pool_load: pivot rows are the fp32 state rounded to binary16,
    bit for bit; integer rows as the quantizer."""
    Hv, Hqk, dk, dv, n_slots, bits = _cases()[case]
    _, S, tb, r, c, codes, pv = _state(case, 600 + case)
    pool = stepq.Pool(n_slots, Hv, Hqk, dk, dv, bits, device=DEV)
    ids = torch.arange(n_slots, dtype=torch.int32, device=DEV)
    pool.load(ids, torch.from_numpy(S).to(DEV), torch.from_numpy(r.reshape(n_slots, Hv, dk)).to(DEV),
              torch.from_numpy(c.reshape(n_slots, Hv, dv)).to(DEV))
    shp = (n_slots, Hv, dk, dv)
    oc = torch.empty(shp, dtype=torch.int8, device=DEV)
    opv = torch.empty(shp, dtype=torch.int16, device=DEV)
    pool.export(ids, oc, torch.empty((n_slots, Hv, dk), device=DEV), torch.empty((n_slots, Hv, dv), device=DEV))
    pool.export_pivots(ids, opv)
    torch.cuda.synchronize()
    assert np.array_equal(opv.cpu().numpy().view(np.uint16).reshape(pv.shape), pv)
    _, y, _ = oracle.quantize(S.reshape(-1, dk, dv).astype(np.float64), r, c, tb, want_y=True)
    PT.compare_codes(oc.cpu().numpy().reshape(codes.shape), codes, y, "pivot pool_load codes")


@pytest.mark.parametrize("mode", [False, True, "row_absmax"])
@pytest.mark.parametrize("kda", [False, True])
@pytest.mark.parametrize("case", range(N_CASES))
def test_pivot_decode_step(case, kda, mode):
    Hv, Hqk, dk, dv, n_slots, bits = _cases()[case]
    _say(f"pivot decode case {case} kda={kda} mode={mode}")
    rng, S, tb, r, c, codes, pv = _state(case, 700 + case)
    pool, all_ids = _pool_with(case, codes, pv, r, c)
    wrow = np.exp(0.3 * rng.standard_normal((Hv, dk))).astype(np.float32)
    pool.set_row_weight(wrow)
    B = max(1, n_slots - 1)
    sel = rng.permutation(n_slots)[:B].astype(np.int32)
    ids = torch.from_numpy(sel).to(DEV)
    q = rng.standard_normal((B, Hqk, dk)); q /= np.linalg.norm(q, axis=-1, keepdims=True)
    k = rng.standard_normal((B, Hqk, dk)); k /= np.linalg.norm(k, axis=-1, keepdims=True)
    v = rng.standard_normal((B, Hv, dv))
    gate = rng.uniform(0.5, 1.0, (B, Hv, dk)) if kda else rng.uniform(0.9, 1.0, (B, Hv))
    be = rng.uniform(0, 1, (B, Hv))
    t32 = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(DEV)
    o = torch.empty((B, Hv, dv), dtype=torch.float32, device=DEV)
    step = pool.step_kda if kda else pool.step
    step(ids, t32(q), t32(k), t32(v), t32(gate), t32(be), o, refit=mode)
    shp = (n_slots, Hv, dk, dv)
    g_codes = torch.empty(shp, dtype=torch.int8, device=DEV)
    g_pv = torch.empty(shp, dtype=torch.int16, device=DEV)
    g_r = torch.empty((n_slots, Hv, dk), device=DEV)
    g_c = torch.empty((n_slots, Hv, dv), device=DEV)
    pool.export(all_ids, g_codes, g_r, g_c)
    pool.export_pivots(all_ids, g_pv)
    torch.cuda.synchronize()
    got = g_codes.cpu().numpy().reshape(-1, dk, dv)
    gpv = g_pv.cpu().numpy().view(np.uint16).reshape(-1, dk, dv)
    gr, gc = g_r.cpu().numpy().reshape(-1, dk), g_c.cpu().numpy().reshape(-1, dv)
    hq = np.arange(Hv) // (Hv // Hqk)
    f32 = lambda a: a.astype(np.float32).astype(np.float64)
    tiles = (sel[:, None] * Hv + np.arange(Hv)[None]).reshape(-1)
    args = (codes[tiles], r[tiles], c[tiles], tb[tiles], f32(q)[:, hq].reshape(-1, dk),
            f32(k)[:, hq].reshape(-1, dk), f32(v).reshape(-1, dv), f32(gate).reshape((-1, dk) if kda else (-1,)),
            f32(be).reshape(-1))
    pmask = tb[tiles] == 16
    if mode is True:
        wt = np.broadcast_to(wrow[None].astype(np.float64), (B, Hv, dk)).reshape(-1, dk)
        new, rn, cn, o_ref, ex, npv = oracle.decode_step_refit(*args, w=wt, want=("y", "c_range"),
                                                               tie_window=PT.TIE_WINDOW, pv=pv[tiles])
        PT.compare_refit(got[tiles], gr[tiles], gc[tiles], new, rn, cn, ex["y"], ex["c_range"], tb[tiles],
                         f"pivot refit case {case}")
        y = ex["y"]
        assert np.array_equal(gr[tiles][pmask], r[tiles][pmask])          # pivots keep their row factor
    elif mode == "row_absmax":
        new, rn, cn, o_ref, y, npv = oracle.decode_step_rowmax(*args, want_y=True, pv=pv[tiles])
        ones = np.ones(cn.shape)
        PT.compare_refit(got[tiles], gr[tiles], gc[tiles], new, rn, cn, y, (ones, ones), tb[tiles],
                         f"pivot row-absmax case {case}")
        assert np.all(gc[tiles] == 1.0)
    else:
        new, o_ref, y, npv = oracle.decode_step(*args, want_y=True, pv=pv[tiles])
        PT.compare_codes(got[tiles], new, y, f"pivot decode case {case}")
        assert np.array_equal(gr[tiles], r[tiles]) and np.array_equal(gc[tiles], c[tiles])
    PT.compare_pivots(gpv[tiles], npv, y, pmask, f"pivot values case {case}")
    PT.compare_out(o.cpu().numpy().reshape(-1, dv), o_ref)
    untouched = np.setdiff1d(np.arange(n_slots * Hv), tiles)
    assert np.array_equal(got[untouched], codes[untouched]) and np.array_equal(gpv[untouched], pv[untouched])


@pytest.mark.parametrize("mode", [False, True, "row_absmax"])
def test_pivot_pool_b512_lockstep(mode):
    """The B=512 pool with pivot rows in a quarter of the heads (the frozen
    and refitting steps run them on the padded uniform bodies in one launch
    with the other heads, the row-absmax step on the generic body), all
    slots stepped, sampled slots compared lockstep."""
    w = W.workload(2)
    bits = row_bits(w)
    bits[W.pivot_mask_draw(w).numpy()] = 16
    PT.lockstep_run(w, 6, np.array([0, 200, 511]), DEV, refit=mode, say=_say, bits=bits)


@pytest.mark.parametrize("mode", [False, True, "row_absmax"])
def test_fp16_heads_pool_b512_lockstep(mode):
    """The B=512 pool with two value heads kept entirely in FP16 (the
    frozen step takes one launch holding the 6-bit, FP16-head and generic
    bodies, the refit one launch of the 6-bit refitting body and the
    FP16-head body, the row-absmax step one launch per class), sampled
    slots compared lockstep."""
    w = W.workload(2)
    bits = row_bits(w)
    bits[W.pivot_head_draw(w, 0, 2).numpy()] = 16
    PT.lockstep_run(w, 4, np.array([0, 311, 511]), DEV, refit=mode, say=_say, bits=bits)


def test_calibrated_map_runs_lockstep():
    """The calibration pipeline (row impact, distortions, lifetime weights,
    pivots, Lagrangian allocation) on the layer_b64 workload's own draws
    yields a map with FP16 pivot rows and 4/8-bit rows; a pool built on it,
    refit with the calibrated row factors, matches the oracle lockstep."""
    from paper_2609_38169_amd.calibrate import calibrate
    w = W.workload(1)
    T = 8
    steps = [W.step_inputs(w, 0, 1000 + t) for t in range(T)]        # calibration draws, not the test steps
    g = w.n_v_heads // w.n_qk_heads
    cat = lambda key: np.concatenate([s[key].numpy() for s in steps])
    q = np.repeat(cat("q"), g, axis=1)
    k = np.repeat(cat("k"), g, axis=1)
    S = W.initial_state(w, 0, range(4)).numpy()
    cal = calibrate(q, k, cat("beta"), cat("alpha"), S, budget=6.0, cand_bits=(4, 8), unit="row",
                    n_pivots=24, horizon=1024)
    bits = cal.row_bits
    assert (bits == 16).sum() == 24 and bits[bits != 16].mean() <= 6.0
    _say(f"calibrated map: {(bits == 8).sum()} rows @8, {(bits == 4).sum()} @4, {(bits == 16).sum()} pivots")
    PT.lockstep_run(w, 8, np.arange(0, 64, 9), DEV, refit=True, row_weight=cal.row_weight, say=_say, bits=bits)


def test_calibrated_head_map_runs_lockstep():
    """The calibration pipeline with head units (the paper's recipe for its
    GDN model: per-head widths by the multiple-choice DP, whole heads kept
    in FP16 as pivots) on the stack48 workload's own draws: the map has
    whole FP16 heads and 4/8-bit heads, and a pool built on it, refit with
    the calibrated row factors, matches the oracle lockstep."""
    from paper_2609_38169_amd.calibrate import calibrate
    w = W.workload(4)
    T = 6
    steps = [W.step_inputs(w, 0, 1000 + t) for t in range(T)]        # calibration draws, not the test steps
    g = w.n_v_heads // w.n_qk_heads
    cat = lambda key: np.concatenate([s[key].float().numpy() for s in steps])
    q = np.repeat(cat("q"), g, axis=1)
    k = np.repeat(cat("k"), g, axis=1)
    S = W.initial_state(w, 0, range(2)).float().numpy()
    cal = calibrate(q, k, cat("beta"), cat("alpha"), S, budget=6.0, cand_bits=(4, 8), unit="head",
                    n_pivots=2, horizon=1024)
    bits = cal.row_bits
    full16 = (bits == 16).all(axis=1)
    assert full16.sum() == 2 and ((bits == 16).any(axis=1) == full16).all()
    per_head = [set(np.unique(b)) for b in bits]
    assert all(len(h) == 1 for h in per_head)                          # one width per head
    assert bits[~full16].mean() <= 6.0
    _say(f"calibrated head map: {int((bits[:, 0] == 8).sum())} heads @8, {int((bits[:, 0] == 4).sum())} @4, "
         f"{int(full16.sum())} FP16 heads")
    PT.lockstep_run(w, 4, np.array([0, 100, 255]), DEV, refit=True, row_weight=cal.row_weight, say=_say, bits=bits)


@pytest.mark.timeout(900)
@pytest.mark.parametrize("refit", [False, True])
def test_calibrated_head_map_pool_b512_every_tile(refit):
    """The head-unit calibrated map that ``bench.py --calibrated head`` times
    (whole heads at 8 or 4 bits and one whole FP16 head, from the
    calibration pipeline on the workload's own draws: the paper's GDN
    setting) at full pool_b512 size, with frozen scales and with the online
    refit: either step is one launch over the compiled bodies of both
    widths (frozen-step or refitting) and the FP16 body, and every tile
    matches the oracle lockstep."""
    from paper_2609_38169_amd.calibrate import calibrate
    w = W.workload(2)
    steps = [W.step_inputs(w, 0, 1000 + t) for t in range(8)]        # calibration draws, not the test steps
    g = w.n_v_heads // w.n_qk_heads
    cat = lambda key: np.concatenate([s[key].float().numpy() for s in steps])
    cal = calibrate(np.repeat(cat("q"), g, axis=1), np.repeat(cat("k"), g, axis=1), cat("beta"), cat("alpha"),
                    W.initial_state(w, 0, range(4)).numpy(), budget=6.0, cand_bits=(4, 8), unit="head",
                    n_pivots=1, horizon=1024)
    bits = cal.row_bits
    full16 = (bits == 16).all(axis=1)
    assert full16.sum() == 1 and all(len(set(np.unique(b))) == 1 for b in bits)
    _say(f"calibrated head map pool_b512: {int((bits[:, 0] == 8).sum())} heads @8, "
         f"{int((bits[:, 0] == 4).sum())} @4, 1 FP16 head")
    PT.lockstep_run(w, 6, np.arange(w.batch), DEV, refit=refit, row_weight=cal.row_weight, say=_say, bits=bits)


@pytest.mark.parametrize("refit", [False, True])
@pytest.mark.parametrize("kind", ["pivot_rows", "fp16_head"])
@pytest.mark.timeout(900)
def test_pivot_maps_pool_b512_every_tile(kind, refit):
    """The maps of ``bench.py --pivots`` (1-3 FP16 pivot rows in a seeded
    quarter of the heads, run by the padded uniform body, frozen-step or
    refitting) and ``bench.py --fp16-heads 1`` (one whole FP16 head beside
    the uniform heads, one combined launch) at full pool_b512 size, with
    frozen scales and with the online refit: every tile lockstep with the
    oracle."""
    from paper_2609_38169_amd.pools import row_bits
    w = W.workload(2)
    bits = row_bits(w).copy()
    if kind == "pivot_rows":
        bits[W.pivot_mask_draw(w).numpy()] = 16
    else:
        bits[W.pivot_head_draw(w, 0, 1).numpy()] = 16
    _say(f"{kind} pool_b512{' refit' if refit else ''}: {int((bits == 16).sum())} FP16 rows")
    PT.lockstep_run(w, 6, np.arange(w.batch), DEV, refit=refit, say=_say, bits=bits)
