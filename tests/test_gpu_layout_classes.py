"""GPU parity on pools whose heads differ in row-width layout.  A pool
spanning every compiled layout and the generic body is advanced with one
launch per layout class (each head's tile found through the launch's head
list), so every class must address its own heads' tiles inside slot records
whose tiles differ in size.  A pool of one uniform layout plus generic heads
takes a single decode launch that holds both bodies.  Frozen, refit and
row-absmax steps, GDN and KDA gates, against the fp64 oracle through the
C ABI."""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_38169_amd import stepq
import _parity as PT

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda", 0)

L1, L2 = {8: 64, 4: 64}, {8: 32, 4: 32, 2: 64}
# rows per width of each head (None: a random {2,4,8} map, the generic body)
MIXES = {
    # the five uniform layouts, a generic mix, then layouts 2 and 1 again, so
    # that classes hold non-adjacent heads: one launch per class
    "all": [L1, L2, {8: 128}, {4: 128}, {2: 128}, None, L2, L1],
    # one uniform layout plus generic heads: one decode launch for both
    "l1_generic": [L1, None, L1, L1, None, L1, L1, L1],
    "l2_generic": [None, L2, L2, L2, L2, L2, L2, None],
}


def _say(*a):
    print(*a, flush=True)


def _bits(rng, mixes):
    rows = []
    for m in mixes:
        if m is None:
            rows.append(rng.choice([2, 4, 8], size=128).astype(np.uint8))
        else:
            rows.append(rng.permutation(np.concatenate([np.full(n, b, np.uint8) for b, n in m.items()])))
    return np.stack(rows)


@pytest.mark.parametrize("levels", [stepq.STEPQ_LEVELS_ABSMAX, stepq.STEPQ_LEVELS_POW2])
@pytest.mark.parametrize("mode", ["frozen", "refit", "row_absmax"])
@pytest.mark.parametrize("kda", [False, True])
@pytest.mark.parametrize("mix", list(MIXES))
def test_layout_classes_one_step(mix, mode, kda, levels):
    Hv, Hqk, dk, dv, n_slots = len(MIXES[mix]), 4, 128, 128, 6
    rng = np.random.default_rng(900 + 100 * list(MIXES).index(mix) + 10 * ["frozen", "refit", "row_absmax"].index(mode)
                                + int(kda) + 1000 * levels)
    bits = _bits(rng, MIXES[mix])
    lv = dict(levels=levels)
    _say(f"layout classes {mix}: mode={mode} kda={kda} levels={levels} Hv={Hv} n_slots={n_slots}")
    S = (rng.standard_normal((n_slots, Hv, dk, dv)) * 0.05).astype(np.float32)
    tb_all = np.broadcast_to(bits[None], (n_slots,) + bits.shape).reshape(-1, dk)
    r, c = oracle.fit_absmax(S.reshape(-1, dk, dv), bits=tb_all, **lv)
    codes = oracle.quantize(S.reshape(-1, dk, dv).astype(np.float64), r, c, tb_all, **lv)
    pool = stepq.Pool(n_slots, Hv, Hqk, dk, dv, bits, device=DEV, levels=levels)
    all_ids = torch.arange(n_slots, dtype=torch.int32, device=DEV)
    pool.import_(all_ids, torch.from_numpy(codes.reshape(n_slots, Hv, dk, dv)).to(DEV),
                 torch.from_numpy(r.reshape(n_slots, Hv, dk)).to(DEV),
                 torch.from_numpy(c.reshape(n_slots, Hv, dv)).to(DEV))
    B = n_slots - 1
    sel = rng.permutation(n_slots)[:B].astype(np.int32)
    ids = torch.from_numpy(sel).to(DEV)
    q = rng.standard_normal((B, Hqk, dk)); q /= np.linalg.norm(q, axis=-1, keepdims=True)
    k = rng.standard_normal((B, Hqk, dk)); k /= np.linalg.norm(k, axis=-1, keepdims=True)
    v = rng.standard_normal((B, Hv, dv))
    gate = rng.uniform(0.5, 1.0, (B, Hv, dk)) if kda else rng.uniform(0.9, 1.0, (B, Hv))
    be = rng.uniform(0, 1, (B, Hv))
    t32 = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(DEV)
    o = torch.empty((B, Hv, dv), dtype=torch.float32, device=DEV)
    refit = {"frozen": False, "refit": True, "row_absmax": "row_absmax"}[mode]
    if kda:
        pool.step_kda(ids, t32(q), t32(k), t32(v), t32(gate), t32(be), o, refit=refit)
    else:
        pool.step(ids, t32(q), t32(k), t32(v), t32(gate), t32(be), o, refit=refit)
    g_codes = torch.empty((n_slots, Hv, dk, dv), dtype=torch.int8, device=DEV)
    g_r = torch.empty((n_slots, Hv, dk), device=DEV)
    g_c = torch.empty((n_slots, Hv, dv), device=DEV)
    pool.export(all_ids, g_codes, g_r, g_c)
    torch.cuda.synchronize()
    got, gr, gc = g_codes.cpu().numpy(), g_r.cpu().numpy(), g_c.cpu().numpy()

    hq = np.arange(Hv) // (Hv // Hqk)
    f32 = lambda a: a.astype(np.float32).astype(np.float64)
    qq, kk = f32(q)[:, hq].reshape(-1, dk), f32(k)[:, hq].reshape(-1, dk)
    vv, bb = f32(v).reshape(-1, dv), f32(be).reshape(-1)
    gt = f32(gate).reshape((-1, dk) if kda else (-1,))
    tiles = (sel[:, None] * Hv + np.arange(Hv)[None]).reshape(-1)
    what = f"layout classes {mix} {mode} kda={kda} levels={levels}"
    gcodes = got.reshape(-1, dk, dv)[tiles]
    if mode == "frozen":
        new, o_ref, y = oracle.decode_step(codes[tiles], r[tiles], c[tiles], tb_all[tiles], qq, kk, vv, gt, bb,
                                           want_y=True, **lv)
        PT.compare_codes(gcodes, new, y, what)
        assert np.array_equal(gr.reshape(-1, dk)[tiles], r[tiles])
        assert np.array_equal(gc.reshape(-1, dv)[tiles], c[tiles])
    elif mode == "refit":
        new, rn, cn, o_ref, ex = oracle.decode_step_refit(codes[tiles], r[tiles], c[tiles], tb_all[tiles], qq, kk,
                                                          vv, gt, bb, want=("y", "c_range"),
                                                          tie_window=PT.TIE_WINDOW, **lv)
        PT.compare_refit(gcodes, gr.reshape(-1, dk)[tiles], gc.reshape(-1, dv)[tiles], new, rn, cn, ex["y"],
                         ex["c_range"], tb_all[tiles], what)
    else:
        new, rn, cn, o_ref, y = oracle.decode_step_rowmax(codes[tiles], r[tiles], c[tiles], tb_all[tiles], qq, kk,
                                                          vv, gt, bb, want_y=True, **lv)
        ones = np.ones(cn.shape)
        PT.compare_refit(gcodes, gr.reshape(-1, dk)[tiles], gc.reshape(-1, dv)[tiles], new, rn, cn, y,
                         (ones, ones), tb_all[tiles], what)
    PT.compare_out(o.cpu().numpy().reshape(-1, dv), o_ref, what + " o")
    # the slot outside the batch keeps its record bit for bit
    for s in np.setdiff1d(np.arange(n_slots), sel):
        assert np.array_equal(got[s], codes.reshape(n_slots, Hv, dk, dv)[s])
        assert np.array_equal(gr[s], r.reshape(n_slots, Hv, dk)[s])
        assert np.array_equal(gc[s], c.reshape(n_slots, Hv, dv)[s])
