"""GPU parity of the decode step with the online dual-axis refit
(stepq_decode_step_ex with STEPQ_STEP_REFIT) against the fp64 oracle,
lockstep, through the C ABI; plus invariants the refit must keep exactly."""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_38169_amd import stepq, workloads as W
from paper_2609_38169_amd.pools import build_pool, row_bits
import _parity as PT

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda", 0)


def _say(*a):
    print(*a, flush=True)


def _run(w, steps, rows, **kw):
    return PT.lockstep_run(w, steps, rows, DEV, refit=True, say=_say, **kw)


def test_refit_tiny_all_steps():
    w = W.workload(0)
    _run(w, w.steps, np.arange(w.batch))


def test_refit_tiny_kda_row_weights():
    w = W.workload(0)
    _run(w, w.steps, np.arange(w.batch), kda=True, row_weight=W.row_weight_draw(w).numpy())


def test_refit_layer_b64_64_steps():
    """Long-lived states (gates near 1): with refit the saturated fraction
    stays small, where frozen scales saturate a large share of codes."""
    w = W.workload(1)
    ls = _run(w, 64, np.arange(w.batch), row_weight=W.row_weight_draw(w).numpy())
    assert ls.saturated < 0.05


@pytest.mark.timeout(900)
@pytest.mark.parametrize("idx", [2, 3])
def test_refit_pool_sized_every_tile(idx):
    """pool_b512 / pool_4bit with the online refit: all 16,384 tiles of the
    full launch compared at every one of 16 steps."""
    w = W.workload(idx)
    ls = _run(w, 16, np.arange(w.batch))
    assert ls.compared == 16 * w.batch * w.n_v_heads * w.d_k * w.d_v


@pytest.mark.timeout(900)
def test_refit_pool_b512_kda_every_tile():
    """Channel-wise gates and row weights with the online refit on the full
    pool_b512 launch, every tile compared for 8 steps."""
    w = W.workload(2)
    _run(w, 8, np.arange(w.batch), kda=True, row_weight=W.row_weight_draw(w).numpy())


def _ragged():
    rng = np.random.default_rng(7)
    cases = []
    for (Hv, Hqk, dk, dv, n_slots) in [(3, 1, 37, 64, 7), (2, 2, 96, 128, 5), (4, 2, 128, 128, 3), (1, 1, 1, 64, 2)]:
        cases.append((Hv, Hqk, dk, dv, n_slots, rng.choice([2, 4, 8], size=(Hv, dk)).astype(np.uint8)))
    cases.append((3, 3, 128, 128, 2, np.stack([np.full(128, b, np.uint8) for b in (8, 4, 2)])))
    return cases


@pytest.mark.parametrize("kda", [False, True])
@pytest.mark.parametrize("case", range(5))
def test_refit_ragged_shapes(case, kda):
    """Generic kernels (irregular width mixes, d_v = 64, d_k not a multiple
    of the group size), random slots, a partial batch, non-uniform w."""
    Hv, Hqk, dk, dv, n_slots, bits = _ragged()[case]
    _say(f"ragged refit case {case} kda={kda}: Hv={Hv} Hqk={Hqk} dk={dk} dv={dv}")
    rng = np.random.default_rng(300 + case)
    S = (rng.standard_normal((n_slots, Hv, dk, dv)) * 0.05).astype(np.float32)
    r, c = oracle.fit_absmax(S.reshape(-1, dk, dv))
    tb_all = np.broadcast_to(bits[None], (n_slots,) + bits.shape).reshape(-1, dk)
    codes = oracle.quantize(S.reshape(-1, dk, dv).astype(np.float64), r, c, tb_all)
    wrow = np.exp(0.4 * rng.standard_normal((Hv, dk))).astype(np.float32)
    pool = stepq.Pool(n_slots, Hv, Hqk, dk, dv, bits, device=DEV)
    pool.set_row_weight(wrow)
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
    gate = rng.uniform(0.5, 1.0, (B, Hv, dk)) if kda else rng.uniform(0.9, 1.0, (B, Hv))
    be = rng.uniform(0, 1, (B, Hv))
    t32 = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(DEV)
    o = torch.empty((B, Hv, dv), dtype=torch.float32, device=DEV)
    if kda:
        pool.step_kda(ids, t32(q), t32(k), t32(v), t32(gate), t32(be), o, refit=True)
    else:
        pool.step(ids, t32(q), t32(k), t32(v), t32(gate), t32(be), o, refit=True)
    g_codes = torch.empty((n_slots, Hv, dk, dv), dtype=torch.int8, device=DEV)
    g_r = torch.empty((n_slots, Hv, dk), device=DEV)
    g_c = torch.empty((n_slots, Hv, dv), device=DEV)
    pool.export(all_ids, g_codes, g_r, g_c)
    torch.cuda.synchronize()
    got, gr, gc = g_codes.cpu().numpy(), g_r.cpu().numpy(), g_c.cpu().numpy()
    hq = np.arange(Hv) // (Hv // Hqk)
    f32 = lambda a: a.astype(np.float32).astype(np.float64)
    qq, kk = f32(q)[:, hq].reshape(-1, dk), f32(k)[:, hq].reshape(-1, dk)
    tiles = (sel[:, None] * Hv + np.arange(Hv)[None]).reshape(-1)
    gt = f32(gate).reshape((-1, dk) if kda else (-1,))
    wt = np.broadcast_to(wrow[None].astype(np.float64), (B, Hv, dk)).reshape(-1, dk)
    new, rn, cn, o_ref, ex = oracle.decode_step_refit(codes[tiles], r[tiles], c[tiles], tb_all[tiles], qq, kk,
                                                      f32(v).reshape(-1, dv), gt, f32(be).reshape(-1), w=wt,
                                                      want=("y", "c_range"), tie_window=PT.TIE_WINDOW)
    PT.compare_refit(got.reshape(-1, dk, dv)[tiles], gr.reshape(-1, dk)[tiles], gc.reshape(-1, dv)[tiles],
                     new, rn, cn, ex["y"], ex["c_range"], tb_all[tiles], f"ragged refit case {case}")
    PT.compare_out(o.cpu().numpy().reshape(-1, dv), o_ref)
    untouched = np.setdiff1d(np.arange(n_slots), sel)
    for s in untouched:
        assert np.array_equal(got[s], codes.reshape(n_slots, Hv, dk, dv)[s])
        assert np.array_equal(gr[s], r.reshape(n_slots, Hv, dk)[s])


def test_refit_power_of_two_weight_invariance():
    """w -> 4 w halves every r' and doubles every c' exactly and leaves the
    codes and the readout unchanged (all the scalings are exact in fp32)."""
    w = W.workload(2)
    bits = row_bits(w)
    pa = build_pool(w, device=DEV, bits=bits)
    pb = stepq.Pool(w.n_slots, w.n_v_heads, w.n_qk_heads, w.d_k, w.d_v, bits, device=DEV)
    pb.memory.copy_(pa.memory)
    wr = W.row_weight_draw(w).numpy()
    pa.set_row_weight(wr)
    pb.set_row_weight(4 * wr)
    ids = W.active_slots(w).to(DEV)
    inp = W.step_inputs(w, 0, 0, device=DEV)
    oa = torch.empty((w.batch, w.n_v_heads, w.d_v), dtype=torch.float32, device=DEV)
    ob = torch.empty_like(oa)
    pa.step(ids, inp["q"], inp["k"], inp["v"], inp["alpha"], inp["beta"], oa, refit=True)
    pb.step(ids, inp["q"], inp["k"], inp["v"], inp["alpha"], inp["beta"], ob, refit=True)
    n = w.batch
    out = []
    for p in (pa, pb):
        cds = torch.empty((n, w.n_v_heads, w.d_k, w.d_v), dtype=torch.int8, device=DEV)
        rr = torch.empty((n, w.n_v_heads, w.d_k), device=DEV)
        cc = torch.empty((n, w.n_v_heads, w.d_v), device=DEV)
        p.export(ids, cds, rr, cc)
        out.append((cds, rr, cc))
    torch.cuda.synchronize()
    assert torch.equal(oa, ob)
    assert torch.equal(out[0][0], out[1][0])
    assert torch.equal(out[0][1], 2 * out[1][1]) and torch.equal(2 * out[0][2], out[1][2])


def test_refit_prepared_call_and_argument_errors():
    w = W.workload(0)
    bits = row_bits(w)
    pa = build_pool(w, device=DEV, bits=bits)
    pb = build_pool(w, device=DEV, bits=bits)
    ids = W.active_slots(w).to(DEV)
    inp = W.step_inputs(w, 0, 0, device=DEV)
    oa = torch.empty((w.batch, w.n_v_heads, w.d_v), dtype=torch.float32, device=DEV)
    ob = torch.empty_like(oa)
    pa.step(ids, inp["q"], inp["k"], inp["v"], inp["alpha"], inp["beta"], oa, refit=True)
    pb.prepare_step(ids, inp["q"], inp["k"], inp["v"], inp["alpha"], inp["beta"], ob, refit=True)()
    torch.cuda.synchronize()
    assert torch.equal(oa, ob) and torch.equal(pa.memory, pb.memory)
    bad = np.ones((w.n_v_heads, w.d_k), np.float32)
    bad[1, 3] = 0.0
    with pytest.raises(stepq.StepqError):
        pa.set_row_weight(bad)
    with pytest.raises(ValueError):
        pa.set_row_weight(np.ones((w.n_v_heads, w.d_k + 1), np.float32))
    with pytest.raises(stepq.StepqError):      # unknown flag bits
        stepq.stepq_decode_step_ex(pa, ids, inp["q"], inp["k"], inp["v"], inp["alpha"], inp["beta"], oa, 16)
