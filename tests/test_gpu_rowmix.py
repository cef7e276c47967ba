"""GPU parity of heads whose integer rows are 8- and 4-bit in any split (the
per-row maps of a row-unit calibration, Section 3.3), stored compact, with
up to 8 FP16 pivot rows: the decode step in all three scale modes, GDN and
KDA, fp32 and bf16 activations, against the fp64 oracle through the C ABI.

No uniform mix holds these heads, so the frozen step runs them on the
row-mix body, whose matrix-core blocks read each word through its slot
views, and the refit on the row-mix refitting body (the same first half,
then the values kept in registers by word-step through the fits).  The split between the 8- and 4-bit row groups is swept across every
position inside a word-step (the groups of one word-step then have
different widths from slice to slice) and across the boundaries of the
4-word groups that form the blocks' K dimension; odd 4-bit row counts leave
an empty slot."""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_38169_amd import stepq
import _parity as PT

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda", 0)


def _say(*a):
    print(*a, flush=True)


def _head(rng, n8, npiv):
    """One head's widths: n8 rows @8, npiv @16, the rest @4, in seeded row order."""
    row = np.concatenate([np.full(n8, 8, np.uint8), np.full(npiv, 16, np.uint8),
                          np.full(128 - n8 - npiv, 4, np.uint8)])
    return rng.permutation(row)


def _cases():
    rng = np.random.default_rng(23)
    cases = []
    # 0: the 8/4 split at every offset in a word-step (n8 mod 8 = 0..7), on
    # both sides of the 32-group block boundaries, odd 4-bit counts; no pivot
    # rows but in the last head
    heads = [(65, 0), (66, 0), (71, 0), (72, 0), (83, 0), (96, 0), (100, 0), (37, 0), (14, 0), (127, 0), (1, 0),
             (33, 2)]
    cases.append((12, 4, 4, np.stack([_head(rng, n8, p) for n8, p in heads])))
    # 1: with 1 to 8 pivot rows (one per slice at most)
    heads = [(70, 3), (30, 8), (90, 5), (100, 1), (65, 2), (20, 7), (96, 4), (81, 6)]
    cases.append((8, 8, 3, np.stack([_head(rng, n8, p) for n8, p in heads])))
    # 2: beside other classes (a 64@8 + 64@4 head, a padded pivot head, a
    # whole FP16 head): one launch per class, GQA 2:1
    b = np.stack([_head(rng, 64, 0), _head(rng, 81, 0), _head(rng, 62, 3), _head(rng, 60, 0)])
    b[3] = 16
    b = np.concatenate([b, np.stack([_head(rng, 64, 0), _head(rng, 77, 2), _head(rng, 88, 0), _head(rng, 50, 2)])])
    cases.append((8, 4, 3, b))
    # 3: 32 heads of seeded random splits (8-bit rows anywhere in 0..128, 0
    # to 8 pivot rows), GQA 4:1: the width boundary and the last group fall
    # at many offsets, and heads that happen to fit a uniform mix take their
    # own class
    hs = []
    for _ in range(32):
        npiv = int(rng.integers(0, 9))
        hs.append(_head(rng, int(rng.integers(0, 129 - npiv)), npiv))
    cases.append((32, 8, 3, np.stack(hs)))
    return cases


N_CASES = 4


def _state(case, seed):
    Hv, Hqk, n_slots, bits = _cases()[case]
    rng = np.random.default_rng(seed)
    S = (rng.standard_normal((n_slots, Hv, 128, 128)) * 0.05).astype(np.float32)
    tb = np.broadcast_to(bits[None], (n_slots,) + bits.shape).reshape(-1, 128)
    r, c = oracle.fit_absmax(S.reshape(-1, 128, 128), bits=tb)
    codes, pv = oracle.quantize(S.reshape(-1, 128, 128).astype(np.float64), r, c, tb)
    return rng, tb, r, c, codes, pv


def _pool_with(case, codes, pv, r, c):
    Hv, Hqk, n_slots, bits = _cases()[case]
    pool = stepq.Pool(n_slots, Hv, Hqk, 128, 128, bits, device=DEV)
    ids = torch.arange(n_slots, dtype=torch.int32, device=DEV)
    pool.import_(ids, torch.from_numpy(codes.reshape(n_slots, Hv, 128, 128)).to(DEV),
                 torch.from_numpy(r.reshape(n_slots, Hv, 128)).to(DEV),
                 torch.from_numpy(c.reshape(n_slots, Hv, 128)).to(DEV))
    pool.import_pivots(ids, torch.from_numpy(pv.reshape(n_slots, Hv, 128, 128).view(np.int16)).to(DEV))
    return pool, ids


@pytest.mark.parametrize("mode", [False, True, "row_absmax"])
@pytest.mark.parametrize("act", ["f32", "bf16"])
@pytest.mark.parametrize("kda", [False, True])
@pytest.mark.parametrize("case", range(N_CASES))
def test_rowmix_decode_step(case, kda, act, mode):
    Hv, Hqk, n_slots, bits = _cases()[case]
    _say(f"row-mix decode case {case} kda={kda} act={act} mode={mode}")
    rng, tb, r, c, codes, pv = _state(case, 800 + case)
    pool, all_ids = _pool_with(case, codes, pv, r, c)
    wrow = np.exp(0.3 * rng.standard_normal((Hv, 128))).astype(np.float32)
    pool.set_row_weight(wrow)
    B = n_slots - 1
    sel = rng.permutation(n_slots)[:B].astype(np.int32)
    ids = torch.from_numpy(sel).to(DEV)
    q = rng.standard_normal((B, Hqk, 128)); q /= np.linalg.norm(q, axis=-1, keepdims=True)
    k = rng.standard_normal((B, Hqk, 128)); k /= np.linalg.norm(k, axis=-1, keepdims=True)
    v = rng.standard_normal((B, Hv, 128))
    gate = rng.uniform(0.5, 1.0, (B, Hv, 128)) if kda else rng.uniform(0.9, 1.0, (B, Hv))
    be = rng.uniform(0, 1, (B, Hv))
    dt = torch.bfloat16 if act == "bf16" else torch.float32
    dev_in = [torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(dt) for a in (q, k, v, gate, be)]
    # the oracle takes the activations exactly as the kernel reads them
    q, k, v, gate, be = (t.float().numpy().astype(np.float64) for t in dev_in)
    o = torch.empty((B, Hv, 128), dtype=torch.float32, device=DEV)
    step = pool.step_kda if kda else pool.step
    step(ids, *(t.to(DEV) for t in dev_in), o, refit=mode)
    shp = (n_slots, Hv, 128, 128)
    g_codes = torch.empty(shp, dtype=torch.int8, device=DEV)
    g_pv = torch.empty(shp, dtype=torch.int16, device=DEV)
    g_r = torch.empty((n_slots, Hv, 128), device=DEV)
    g_c = torch.empty((n_slots, Hv, 128), device=DEV)
    pool.export(all_ids, g_codes, g_r, g_c)
    pool.export_pivots(all_ids, g_pv)
    torch.cuda.synchronize()
    got = g_codes.cpu().numpy().reshape(-1, 128, 128)
    gpv = g_pv.cpu().numpy().view(np.uint16).reshape(-1, 128, 128)
    gr, gc = g_r.cpu().numpy().reshape(-1, 128), g_c.cpu().numpy().reshape(-1, 128)
    hq = np.arange(Hv) // (Hv // Hqk)
    tiles = (sel[:, None] * Hv + np.arange(Hv)[None]).reshape(-1)
    args = (codes[tiles], r[tiles], c[tiles], tb[tiles], q[:, hq].reshape(-1, 128), k[:, hq].reshape(-1, 128),
            v.reshape(-1, 128), gate.reshape((-1, 128) if kda else (-1,)), be.reshape(-1))
    pmask = tb[tiles] == 16
    if mode is True:
        wt = np.broadcast_to(wrow[None].astype(np.float64), (B, Hv, 128)).reshape(-1, 128)
        new, rn, cn, o_ref, ex, npv = oracle.decode_step_refit(*args, w=wt, want=("y", "c_range"),
                                                               tie_window=PT.TIE_WINDOW, pv=pv[tiles])
        PT.compare_refit(got[tiles], gr[tiles], gc[tiles], new, rn, cn, ex["y"], ex["c_range"], tb[tiles],
                         f"row-mix refit case {case}")
        y = ex["y"]
    elif mode == "row_absmax":
        new, rn, cn, o_ref, y, npv = oracle.decode_step_rowmax(*args, want_y=True, pv=pv[tiles])
        ones = np.ones(cn.shape)
        PT.compare_refit(got[tiles], gr[tiles], gc[tiles], new, rn, cn, y, (ones, ones), tb[tiles],
                         f"row-mix row-absmax case {case}")
    else:
        new, o_ref, y, npv = oracle.decode_step(*args, want_y=True, pv=pv[tiles])
        PT.compare_codes(got[tiles], new, y, f"row-mix decode case {case}")
        assert np.array_equal(gr[tiles], r[tiles]) and np.array_equal(gc[tiles], c[tiles])
    PT.compare_pivots(gpv[tiles], npv, y, pmask, f"row-mix pivot values case {case}")
    PT.compare_out(o.cpu().numpy().reshape(-1, 128), o_ref)
    # slots outside the batch are untouched
    rest = np.setdiff1d(np.arange(n_slots), sel)
    rt = (rest[:, None] * Hv + np.arange(Hv)[None]).reshape(-1)
    assert np.array_equal(got[rt], codes[rt]) and np.array_equal(gpv[rt], pv[rt])


def test_rowmix_lockstep_steps():
    """Several frozen steps in lockstep on case 1 (pivot heads): each step is
    checked against the oracle run from the GPU's own stored input."""
    Hv, Hqk, n_slots, bits = _cases()[1]
    _say("row-mix lockstep case 1")
    rng, tb, r, c, codes, pv = _state(1, 900)
    pool, ids = _pool_with(1, codes, pv, r, c)
    shp = (n_slots, Hv, 128, 128)
    hq = np.arange(Hv) // (Hv // Hqk)
    for step in range(4):
        g_codes = torch.empty(shp, dtype=torch.int8, device=DEV)
        g_pv = torch.empty(shp, dtype=torch.int16, device=DEV)
        pool.export(ids, g_codes, torch.empty((n_slots, Hv, 128), device=DEV),
                    torch.empty((n_slots, Hv, 128), device=DEV))
        pool.export_pivots(ids, g_pv)
        q = rng.standard_normal((n_slots, Hqk, 128)); q /= np.linalg.norm(q, axis=-1, keepdims=True)
        k = rng.standard_normal((n_slots, Hqk, 128)); k /= np.linalg.norm(k, axis=-1, keepdims=True)
        v = rng.standard_normal((n_slots, Hv, 128))
        al = rng.uniform(0.9, 1.0, (n_slots, Hv))
        be = rng.uniform(0, 1, (n_slots, Hv))
        q, k, v, al, be = (a.astype(np.float32).astype(np.float64) for a in (q, k, v, al, be))
        t32 = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(DEV)
        o = torch.empty((n_slots, Hv, 128), dtype=torch.float32, device=DEV)
        pool.step(ids, t32(q), t32(k), t32(v), t32(al), t32(be), o)
        n_codes = torch.empty(shp, dtype=torch.int8, device=DEV)
        n_pv = torch.empty(shp, dtype=torch.int16, device=DEV)
        pool.export(ids, n_codes, torch.empty((n_slots, Hv, 128), device=DEV),
                    torch.empty((n_slots, Hv, 128), device=DEV))
        pool.export_pivots(ids, n_pv)
        torch.cuda.synchronize()
        cin = g_codes.cpu().numpy().reshape(-1, 128, 128)
        pin = g_pv.cpu().numpy().view(np.uint16).reshape(-1, 128, 128)
        new, o_ref, y, npv = oracle.decode_step(cin, r, c, tb, q[:, hq].reshape(-1, 128), k[:, hq].reshape(-1, 128),
                                                v.reshape(-1, 128), al.reshape(-1), be.reshape(-1), want_y=True,
                                                pv=pin)
        PT.compare_codes(n_codes.cpu().numpy().reshape(-1, 128, 128), new, y, f"row-mix lockstep step {step}")
        PT.compare_pivots(n_pv.cpu().numpy().view(np.uint16).reshape(-1, 128, 128), npv, y, tb == 16,
                          f"row-mix lockstep pivots step {step}")
        PT.compare_out(o.cpu().numpy().reshape(-1, 128), o_ref)


def _calibrated_row_map():
    """The row-unit calibrated map that ``bench.py --calibrated row`` times
    (per-head 8/4-bit splits, 24 FP16 pivot rows, from the calibration
    pipeline on the workload's own draws) and its row-impact factors."""
    from paper_2609_38169_amd import workloads as W
    from paper_2609_38169_amd.calibrate import calibrate
    w = W.workload(2)
    draws = [W.step_inputs(w, 0, 1000 + t) for t in range(8)]          # calibration draws, not the test steps
    g = w.n_v_heads // w.n_qk_heads
    cat = lambda key: np.concatenate([d[key].float().numpy() for d in draws])
    cal = calibrate(np.repeat(cat("q"), g, axis=1), np.repeat(cat("k"), g, axis=1), cat("beta"), cat("alpha"),
                    W.initial_state(w, 0, range(4)).numpy(), budget=6.0, cand_bits=(4, 8), unit="row",
                    n_pivots=24, horizon=1024)
    bits = cal.row_bits
    n16 = (bits == 16).sum(1)
    assert n16.sum() == 24 and n16.max() <= 8 and not (bits == 2).any()
    _say(f"row-unit calibrated pool_b512: {(bits == 8).sum()} rows @8, {(bits == 4).sum()} @4, 24 pivots")
    return w, bits, cal.row_weight


@pytest.mark.timeout(900)
@pytest.mark.parametrize("kda", [False, True])
def test_rowmix_calibrated_pool_b512_every_tile(kda):
    """The row-unit calibrated map at full pool_b512 size, in the launch
    configuration ``bench.py --calibrated row`` times, with the scalar gate
    and with channel-wise (KDA) gates: every tile lockstep with the oracle
    over several frozen steps."""
    w, bits, row_weight = _calibrated_row_map()
    PT.lockstep_run(w, 6, np.arange(w.batch), DEV, row_weight=row_weight, say=_say, bits=bits, kda=kda)


@pytest.mark.timeout(900)
@pytest.mark.parametrize("kda,levels", [(True, 1), (False, 0)])
def test_rowmix_calibrated_refit_pool_b512_every_tile(kda, levels):
    """The decode step with the online dual-axis refit on the row-unit
    calibrated map at full pool_b512 size (the row-mix refitting body), as
    ``bench.py --calibrated row --refit`` times it: channel-wise gates on the
    2^(8-b) q codebook (the paper's KDA setting: row-level allocation, FP16
    pivot rows, the shared column fit over the mixed-width integer rows) and
    the scalar gate on q / q_b levels.  Every tile lockstep with the oracle
    over several steps."""
    w, bits, row_weight = _calibrated_row_map()
    PT.lockstep_run(w, 6, np.arange(w.batch), DEV, refit=True, row_weight=row_weight, say=_say, bits=bits,
                    kda=kda, levels=levels)


@pytest.mark.timeout(900)
def test_rowmix_kda_setting_refit_64_steps():
    """The paper's KDA decode step (row-unit calibrated map with FP16 pivot
    rows, channel-wise gates on the 2^(8-b) q codebook, the dual-axis refit
    every step) over 64 steps of the full pool_b512 launch: a third of the
    requests (every head) lockstep with the oracle at every step."""
    w, bits, row_weight = _calibrated_row_map()
    PT.lockstep_run(w, 64, np.arange(0, w.batch, 3), DEV, refit=True, row_weight=row_weight, say=_say, bits=bits,
                    kda=True, levels=1)
