"""GPU parity of the decode step with the row-wise absmax requantization of
the INT-b baseline (stepq_decode_step_ex with STEPQ_STEP_ROW_ABSMAX) against
the fp64 oracle, lockstep, through the C ABI."""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_38169_amd import stepq, workloads as W
import _parity as PT

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda", 0)


def _say(*a):
    print(*a, flush=True)


def _run(w, steps, rows, **kw):
    return PT.lockstep_run(w, steps, rows, DEV, refit="row_absmax", say=_say, **kw)


def test_rowmax_tiny_all_steps():
    w = W.workload(0)
    _run(w, w.steps, np.arange(w.batch))


def test_rowmax_layer_b64_64_steps():
    w = W.workload(1)
    _run(w, 64, np.arange(w.batch))


@pytest.mark.timeout(900)
@pytest.mark.parametrize("idx", [2, 3])
def test_rowmax_pool_sized_every_tile(idx):
    """pool_b512 / pool_4bit with the row-absmax step: all 16,384 tiles of
    the full launch compared at every one of 16 steps."""
    w = W.workload(idx)
    ls = _run(w, 16, np.arange(w.batch))
    assert ls.compared == 16 * w.batch * w.n_v_heads * w.d_k * w.d_v


@pytest.mark.timeout(900)
def test_rowmax_pool_b512_kda_every_tile():
    w = W.workload(2)
    _run(w, 8, np.arange(w.batch), kda=True)


@pytest.mark.parametrize("case", range(5))
def test_rowmax_ragged_shapes(case):
    """Generic kernels: irregular width mixes, d_v = 64, ragged d_k."""
    rng = np.random.default_rng(7)
    cases = []
    for (Hv, Hqk, dk, dv, n_slots) in [(3, 1, 37, 64, 7), (2, 2, 96, 128, 5), (4, 2, 128, 128, 3), (1, 1, 1, 64, 2)]:
        cases.append((Hv, Hqk, dk, dv, n_slots, rng.choice([2, 4, 8], size=(Hv, dk)).astype(np.uint8)))
    cases.append((3, 3, 128, 128, 2, np.stack([np.full(128, b, np.uint8) for b in (8, 4, 2)])))
    Hv, Hqk, dk, dv, n_slots, bits = cases[case]
    _say(f"ragged row-absmax case {case}: Hv={Hv} Hqk={Hqk} dk={dk} dv={dv}")
    rng = np.random.default_rng(400 + case)
    S = (rng.standard_normal((n_slots, Hv, dk, dv)) * 0.05).astype(np.float32)
    r, c = oracle.fit_absmax(S.reshape(-1, dk, dv))
    tb_all = np.broadcast_to(bits[None], (n_slots,) + bits.shape).reshape(-1, dk)
    codes = oracle.quantize(S.reshape(-1, dk, dv).astype(np.float64), r, c, tb_all)
    pool = stepq.Pool(n_slots, Hv, Hqk, dk, dv, bits, device=DEV)
    all_ids = torch.arange(n_slots, dtype=torch.int32, device=DEV)
    pool.import_(all_ids, torch.from_numpy(codes.reshape(n_slots, Hv, dk, dv)).to(DEV),
                 torch.from_numpy(r.reshape(n_slots, Hv, dk)).to(DEV),
                 torch.from_numpy(c.reshape(n_slots, Hv, dv)).to(DEV))
    B = max(1, n_slots - 1)
    sel = rng.permutation(n_slots)[:B].astype(np.int32)
    ids = torch.from_numpy(sel).to(DEV)
    q = rng.standard_normal((B, Hqk, dk)); q /= np.linalg.norm(q, axis=-1, keepdims=True)
    k = rng.standard_normal((B, Hqk, dk)); k /= np.linalg.norm(k, axis=-1, keepdims=True)
    v = rng.standard_normal((B, Hv, dv))
    al = rng.uniform(0.9, 1.0, (B, Hv)); be = rng.uniform(0, 1, (B, Hv))
    t32 = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(DEV)
    o = torch.empty((B, Hv, dv), dtype=torch.float32, device=DEV)
    pool.step(ids, t32(q), t32(k), t32(v), t32(al), t32(be), o, refit="row_absmax")
    g_codes = torch.empty((n_slots, Hv, dk, dv), dtype=torch.int8, device=DEV)
    g_r = torch.empty((n_slots, Hv, dk), device=DEV)
    g_c = torch.empty((n_slots, Hv, dv), device=DEV)
    pool.export(all_ids, g_codes, g_r, g_c)
    torch.cuda.synchronize()
    got, gr, gc = g_codes.cpu().numpy(), g_r.cpu().numpy(), g_c.cpu().numpy()
    hq = np.arange(Hv) // (Hv // Hqk)
    f32 = lambda a: a.astype(np.float32).astype(np.float64)
    tiles = (sel[:, None] * Hv + np.arange(Hv)[None]).reshape(-1)
    new, rn, cn, o_ref, y = oracle.decode_step_rowmax(codes[tiles], r[tiles], c[tiles], tb_all[tiles],
                                                      f32(q)[:, hq].reshape(-1, dk), f32(k)[:, hq].reshape(-1, dk),
                                                      f32(v).reshape(-1, dv), f32(al).reshape(-1),
                                                      f32(be).reshape(-1), want_y=True)
    assert np.all(gc.reshape(-1, dv)[tiles] == 1.0)
    ones = np.ones(cn.shape)
    PT.compare_refit(got.reshape(-1, dk, dv)[tiles], gr.reshape(-1, dk)[tiles], gc.reshape(-1, dv)[tiles],
                     new, rn, cn, y, (ones, ones), tb_all[tiles], f"ragged row-absmax case {case}")
    PT.compare_out(o.cpu().numpy().reshape(-1, dv), o_ref)
    for s in np.setdiff1d(np.arange(n_slots), sel):
        assert np.array_equal(got[s], codes.reshape(n_slots, Hv, dk, dv)[s])


def test_rowmax_flag_errors():
    w = W.workload(0)
    from paper_2609_38169_amd.pools import build_pool, row_bits
    pool = build_pool(w, device=DEV, bits=row_bits(w))
    ids = W.active_slots(w).to(DEV)
    inp = W.step_inputs(w, 0, 0, device=DEV)
    o = torch.empty((w.batch, w.n_v_heads, w.d_v), dtype=torch.float32, device=DEV)
    with pytest.raises(stepq.StepqError):     # the two refits exclude each other
        stepq.stepq_decode_step_ex(pool, ids, inp["q"], inp["k"], inp["v"], inp["alpha"], inp["beta"], o,
                                   stepq.STEPQ_STEP_REFIT | stepq.STEPQ_STEP_ROW_ABSMAX)
    with pytest.raises(ValueError):
        pool.step(ids, inp["q"], inp["k"], inp["v"], inp["alpha"], inp["beta"], o, refit="rowmax")
