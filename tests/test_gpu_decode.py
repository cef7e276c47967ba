"""GPU parity of the HIP path against the fp64 oracle, through the C ABI.

Every workload runs the full launch (every active slot, the configuration
bench.py times) and is checked on every tile, lockstep (see
tests/_parity.py): tiny for all of its 32 steps, layer_b64, pool_b512 and
pool_4bit for 64 steps, stack48 on all requests of layers 0, 23 and 47 for
64 graph replays.
"""
import os

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


def _ragged_cases():
    rng = np.random.default_rng(7)
    cases = []
    for (Hv, Hqk, dk, dv, n_slots) in [(3, 1, 37, 64, 7), (2, 2, 96, 128, 5), (4, 2, 128, 128, 3), (1, 1, 1, 64, 2)]:
        bits = rng.choice([2, 4, 8], size=(Hv, dk)).astype(np.uint8)
        cases.append((Hv, Hqk, dk, dv, n_slots, bits))
    # whole-width heads
    cases.append((3, 3, 128, 128, 2, np.stack([np.full(128, b, np.uint8) for b in (8, 4, 2)])))
    return cases


@pytest.mark.parametrize("case", range(5))
def test_import_export_bit_exact(case):
    Hv, Hqk, dk, dv, n_slots, bits = _ragged_cases()[case]
    _say(f"import/export case {case}: Hv={Hv} dk={dk} dv={dv}")
    rng = np.random.default_rng(case)
    qb = 2 ** (bits.astype(np.int64) - 1) - 1
    codes = rng.integers(-qb[None, :, :, None], qb[None, :, :, None] + 1, size=(n_slots, Hv, dk, dv)).astype(np.int8)
    r = rng.uniform(0.01, 1, (n_slots, Hv, dk)).astype(np.float32)
    c = rng.uniform(0.01, 1, (n_slots, Hv, dv)).astype(np.float32)
    pool = stepq.Pool(n_slots, Hv, Hqk, dk, dv, bits, device=DEV)
    pool.memory.fill_(0xA5)            # padding must come out zero
    perm = rng.permutation(n_slots).astype(np.int32)
    ids = torch.from_numpy(perm).to(DEV)
    pool.import_(ids, torch.from_numpy(codes[perm]).to(DEV), torch.from_numpy(r[perm]).to(DEV),
                 torch.from_numpy(c[perm]).to(DEV))
    img = pool.memory.cpu().numpy()
    assert np.array_equal(img, oracle.pack_pool(codes, r, c, bits)), "pool image differs from the layout definition"
    oc = torch.empty((n_slots, Hv, dk, dv), dtype=torch.int8, device=DEV)
    orr = torch.empty((n_slots, Hv, dk), dtype=torch.float32, device=DEV)
    occ = torch.empty((n_slots, Hv, dv), dtype=torch.float32, device=DEV)
    pool.export(ids, oc, orr, occ)
    assert np.array_equal(oc.cpu().numpy(), codes[perm])
    assert np.array_equal(orr.cpu().numpy(), r[perm]) and np.array_equal(occ.cpu().numpy(), c[perm])
    # dequantization: fp32 against fp64, well inside one level
    deq = torch.empty((n_slots, Hv, dk, dv), dtype=torch.float32, device=DEV)
    pool.dequant(ids, deq)
    ref = oracle.dequant(codes.reshape(-1, dk, dv), r.reshape(-1, dk), c.reshape(-1, dv),
                         np.broadcast_to(bits[None], (n_slots,) + bits.shape).reshape(-1, dk)).reshape(codes.shape)
    lsb = (r.astype(np.float64)[..., None] * c.astype(np.float64)[:, :, None, :]) / qb[None, :, :, None]
    err = np.abs(deq.cpu().numpy()[np.argsort(perm)] - ref)
    assert np.all(err <= 1e-3 * lsb)


@pytest.mark.parametrize("idx", [0, 3])
def test_pool_load_matches_oracle_quantizer(idx):
    w = W.workload(idx)
    n = min(w.n_slots, 8)
    _say(f"pool_load workload {w.name}: {n} slots")
    bits = row_bits(w)
    S = W.initial_state(w, 0, range(n), device=DEV)
    r, c = stepq.stepq_setup_fit(S.cpu())
    pool = stepq.Pool(n, w.n_v_heads, w.n_qk_heads, w.d_k, w.d_v, bits, device=DEV)
    ids = torch.arange(n, dtype=torch.int32, device=DEV)
    pool.load(ids, S, torch.from_numpy(r).to(DEV), torch.from_numpy(c).to(DEV))
    codes = torch.empty((n, w.n_v_heads, w.d_k, w.d_v), dtype=torch.int8, device=DEV)
    pool.export(ids, codes, torch.empty_like(torch.from_numpy(r)).to(DEV), torch.empty_like(torch.from_numpy(c)).to(DEV))
    Sn = S.cpu().numpy().reshape(-1, w.d_k, w.d_v)
    ro, co = oracle.fit_absmax(Sn)
    tb = np.broadcast_to(bits[None], (n,) + bits.shape).reshape(-1, w.d_k)
    oc, y = oracle.quantize(Sn.astype(np.float64), ro, co, tb, want_y=True)
    PT.compare_codes(codes.cpu().numpy().reshape(oc.shape), oc, y, "pool_load codes")


def _lockstep_run(w, steps, check_rows, layer=0, mutate=None, kda=False):
    return PT.lockstep_run(w, steps, check_rows, DEV, layer=layer, mutate=mutate, kda=kda, say=_say)


def test_decode_tiny_all_steps():
    w = W.workload(0)
    _lockstep_run(w, w.steps, np.arange(w.batch))


def test_decode_layer_b64_64_steps():
    w = W.workload(1)
    _lockstep_run(w, 64, np.arange(w.batch))


@pytest.mark.timeout(900)
@pytest.mark.parametrize("idx", [2, 3])
def test_decode_pool_sized_every_tile(idx):
    """pool_b512 / pool_4bit: all 512 requests x 32 heads (16,384 tiles) of
    the full launch compared at every one of 64 steps."""
    w = W.workload(idx)
    ls = _lockstep_run(w, 64, np.arange(w.batch))
    assert ls.compared == 64 * w.batch * w.n_v_heads * w.d_k * w.d_v


def test_identity_gate_keeps_codes():
    """alpha = 1, beta = 0: X = S^, so every code comes back unchanged and
    o = S^T q (exact in code space on the GPU as well)."""
    w = W.workload(0)
    bits = row_bits(w)
    pool = build_pool(w, device=DEV, bits=bits)
    ids = W.active_slots(w).to(DEV)
    n = w.batch
    before = torch.empty((n, w.n_v_heads, w.d_k, w.d_v), dtype=torch.int8, device=DEV)
    rr = torch.empty((n, w.n_v_heads, w.d_k), dtype=torch.float32, device=DEV)
    cc = torch.empty((n, w.n_v_heads, w.d_v), dtype=torch.float32, device=DEV)
    pool.export(ids, before, rr, cc)
    inp = W.step_inputs(w, 0, 0, device=DEV)
    inp["alpha"] = torch.ones_like(inp["alpha"])
    inp["beta"] = torch.zeros_like(inp["beta"])
    o = torch.empty((n, w.n_v_heads, w.d_v), dtype=torch.float32, device=DEV)
    pool.step(ids, inp["q"], inp["k"], inp["v"], inp["alpha"], inp["beta"], o)
    after = torch.empty_like(before)
    pool.export(ids, after, rr, cc)
    assert torch.equal(before, after)
    deq = torch.empty((n, w.n_v_heads, w.d_k, w.d_v), dtype=torch.float32, device=DEV)
    pool.dequant(ids, deq)
    ref = torch.einsum("bhij,bhi->bhj", deq.double().cpu(), inp["q"].double().cpu())
    assert torch.allclose(o.double().cpu(), ref, rtol=1e-5, atol=1e-6)


def test_full_write_recalls_value():
    """alpha = beta = 1, q := k with |k| = 1: X^T k = v before requantization,
    so the readout returns v."""
    w = W.workload(1)
    bits = row_bits(w)
    pool = build_pool(w, device=DEV, bits=bits)
    ids = W.active_slots(w).to(DEV)
    inp = W.step_inputs(w, 0, 0, device=DEV)
    o = torch.empty((w.batch, w.n_v_heads, w.d_v), dtype=torch.float32, device=DEV)
    pool.step(ids, inp["k"], inp["k"], inp["v"], torch.ones_like(inp["alpha"]), torch.ones_like(inp["beta"]), o)
    torch.cuda.synchronize()
    assert torch.allclose(o, inp["v"], rtol=0, atol=2e-5)


@pytest.mark.parametrize("case", range(5))
def test_decode_ragged_shapes(case):
    """Odd row counts per width (empty group slots), d_k not a multiple of the
    group size, d_v = 64, GQA 3:1, random slot ids, a partial batch."""
    Hv, Hqk, dk, dv, n_slots, bits = _ragged_cases()[case]
    _say(f"ragged decode case {case}: Hv={Hv} Hqk={Hqk} dk={dk} dv={dv}")
    rng = np.random.default_rng(100 + case)
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
    pool.step(ids, t32(q), t32(k), t32(v), t32(al), t32(be), o)
    out = torch.empty((n_slots, Hv, dk, dv), dtype=torch.int8, device=DEV)
    pool.export(all_ids, out, torch.empty((n_slots, Hv, dk), device=DEV), torch.empty((n_slots, Hv, dv), device=DEV))
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    hq = np.arange(Hv) // (Hv // Hqk)
    f32 = lambda a: a.astype(np.float32).astype(np.float64)
    qq, kk = f32(q)[:, hq].reshape(-1, dk), f32(k)[:, hq].reshape(-1, dk)
    tiles = (sel[:, None] * Hv + np.arange(Hv)[None]).reshape(-1)
    new, o_ref, y = oracle.decode_step(codes[tiles], r[tiles], c[tiles], tb_all[tiles], qq, kk,
                                       f32(v).reshape(-1, dv), f32(al).reshape(-1), f32(be).reshape(-1), want_y=True)
    PT.compare_codes(got.reshape(-1, dk, dv)[tiles], new, y, f"ragged case {case}")
    PT.compare_out(o.cpu().numpy().reshape(-1, dv), o_ref)
    untouched = np.setdiff1d(np.arange(n_slots), sel)
    for s in untouched:
        assert np.array_equal(got[s], codes.reshape(n_slots, Hv, dk, dv)[s])


def test_batch_zero_and_argument_errors(monkeypatch):
    w = W.workload(0)
    pool = stepq.Pool(2, w.n_v_heads, w.n_qk_heads, w.d_k, w.d_v, row_bits(w), device=DEV)
    z = lambda *s, dt=torch.float32: torch.zeros(s, dtype=dt, device=DEV)
    ids0 = torch.zeros(0, dtype=torch.int32, device=DEV)
    pool.step(ids0, z(0, 4, 64), z(0, 4, 64), z(0, 4, 64), z(0, 4), z(0, 4), z(0, 4, 64))
    ids = torch.tensor([0, 1], dtype=torch.int32, device=DEV)
    with pytest.raises(ValueError):          # wrong v shape: caught before any launch
        pool.step(ids, z(2, 4, 64), z(2, 4, 64), z(2, 4, 32), z(2, 4), z(2, 4), z(2, 4, 64))
    with pytest.raises(TypeError):
        pool.step(ids, z(2, 4, 64), z(2, 4, 64), z(2, 4, 64), z(2, 4), z(2, 4), z(2, 4, 64, dt=torch.float16))
    monkeypatch.setenv("STEPQ_DEBUG", "1")
    dup = torch.tensor([1, 1], dtype=torch.int32, device=DEV)
    with pytest.raises(stepq.StepqError) as e:
        pool.step(dup, z(2, 4, 64), z(2, 4, 64), z(2, 4, 64), z(2, 4), z(2, 4), z(2, 4, 64))
    assert e.value.status == 1
    oob = torch.tensor([0, 5], dtype=torch.int32, device=DEV)
    with pytest.raises(stepq.StepqError):
        pool.step(oob, z(2, 4, 64), z(2, 4, 64), z(2, 4, 64), z(2, 4), z(2, 4), z(2, 4, 64))
    too_many = torch.zeros(3, dtype=torch.int32, device=DEV)
    monkeypatch.delenv("STEPQ_DEBUG")
    with pytest.raises(stepq.StepqError):
        pool.step(too_many, z(3, 4, 64), z(3, 4, 64), z(3, 4, 64), z(3, 4), z(3, 4), z(3, 4, 64))


@pytest.mark.timeout(900)
def test_decode_stack48_graph():
    """48 layers, one launch per layer captured once in a HIP graph and
    replayed per decode step; every request of layers 0, 23 and 47 checked
    lockstep at each of 64 replays, with eager imports/exports between
    replays."""
    w = W.workload(4)
    steps, rows, layers_checked = 64, np.arange(w.batch), (0, 23, 47)
    slots = W.active_slots(w).to(DEV)
    pools, locks, bufs = [], {}, []
    for L in range(w.layers):
        bits = row_bits(w, L)
        pools.append(build_pool(w, L, device=DEV, bits=bits))
        if L in layers_checked:
            S0 = W.initial_state(w, L, [int(s) for s in W.active_slots(w)[rows]], device=DEV).cpu().numpy()
            locks[L] = PT.Lockstep(w, pools[L], slots, bits, rows, S0, L)
        inp = W.step_inputs(w, L, 0, device=DEV)
        bufs.append({k: v.clone() for k, v in inp.items()})
        bufs[L]["o"] = torch.empty((w.batch, w.n_v_heads, w.d_v), dtype=torch.float32, device=DEV)
        if L % 8 == 7:
            _say(f"stack48: {L + 1} layer pools built")
    _say("stack48: pools built, capturing")
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        with torch.cuda.graph(graph, stream=side):
            for L in range(w.layers):
                b = bufs[L]
                pools[L].step(slots, b["q"], b["k"], b["v"], b["alpha"], b["beta"], b["o"])
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    for t in range(steps):
        step_inp = {}
        for L in range(w.layers):
            inp = W.step_inputs(w, L, t, device=DEV)
            for key in inp:
                bufs[L][key].copy_(inp[key])
            if L in layers_checked:
                step_inp[L] = inp
                locks[L].anchor()
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for L in layers_checked:
            locks[L].check_step(step_inp[L], bufs[L]["o"], t)
        if t % 8 == 7:
            _say(f"stack48: replay {t} ok")
    for L in layers_checked:
        locks[L].finish(f"stack48 layer {L}")
        assert locks[L].compared == steps * w.batch * w.n_v_heads * w.d_k * w.d_v
        _say(f"stack48 layer {L}: {locks[L].mismatches} code mismatches of {locks[L].compared}")


def test_prepared_step_matches_checked_call():
    """Pool.prepare_step launches the same C call with cached arguments."""
    w = W.workload(0)
    bits = row_bits(w)
    pa = build_pool(w, device=DEV, bits=bits)
    pb = build_pool(w, device=DEV, bits=bits)
    ids = W.active_slots(w).to(DEV)
    inp = W.step_inputs(w, 0, 0, device=DEV)
    oa = torch.empty((w.batch, w.n_v_heads, w.d_v), dtype=torch.float32, device=DEV)
    ob = torch.empty_like(oa)
    pa.step(ids, inp["q"], inp["k"], inp["v"], inp["alpha"], inp["beta"], oa)
    run = pb.prepare_step(ids, inp["q"], inp["k"], inp["v"], inp["alpha"], inp["beta"], ob)
    run()
    torch.cuda.synchronize()
    assert torch.equal(oa, ob) and torch.equal(pa.memory, pb.memory)


# --- KDA: channel-wise retention gate D = diag(d) -----------------------------

def test_kda_tiny_all_steps():
    w = W.workload(0)
    _lockstep_run(w, w.steps, np.arange(w.batch), kda=True)


def test_kda_layer_b64_64_steps():
    w = W.workload(1)
    _lockstep_run(w, 64, np.arange(w.batch), kda=True)


@pytest.mark.timeout(900)
@pytest.mark.parametrize("idx", [2, 3])
def test_kda_pool_sized_every_tile(idx):
    """Channel-wise gates on the full pool_b512 / pool_4bit launch, every
    tile compared for 16 steps."""
    w = W.workload(idx)
    _lockstep_run(w, 16, np.arange(w.batch), kda=True)


def test_kda_identity_gate_keeps_codes():
    """d = 1 on every row and beta = 0: X = S^, codes come back unchanged."""
    w = W.workload(1)
    bits = row_bits(w)
    pool = build_pool(w, device=DEV, bits=bits)
    ids = W.active_slots(w).to(DEV)
    before = pool.memory.clone()
    inp = W.step_inputs(w, 0, 0, device=DEV)
    o = torch.empty((w.batch, w.n_v_heads, w.d_v), dtype=torch.float32, device=DEV)
    gate = torch.ones((w.batch, w.n_v_heads, w.d_k), dtype=inp["alpha"].dtype, device=DEV)
    pool.step_kda(ids, inp["q"], inp["k"], inp["v"], gate, torch.zeros_like(inp["beta"]), o)
    torch.cuda.synchronize()
    assert torch.equal(before, pool.memory)


def test_kda_uniform_gate_matches_gdn_call():
    """d_i = alpha for every row: the KDA call and the GDN call compute the
    same update (they fold the gate at different points, so codes may differ
    only at rounding ties and o within the output tolerance)."""
    w = W.workload(2)
    bits = row_bits(w)
    pa = build_pool(w, device=DEV, bits=bits)
    pb = stepq.Pool(w.n_slots, w.n_v_heads, w.n_qk_heads, w.d_k, w.d_v, bits, device=DEV)
    pb.memory.copy_(pa.memory)
    ids = W.active_slots(w).to(DEV)
    inp = W.step_inputs(w, 0, 0, device=DEV)
    oa = torch.empty((w.batch, w.n_v_heads, w.d_v), dtype=torch.float32, device=DEV)
    ob = torch.empty_like(oa)
    pa.step(ids, inp["q"], inp["k"], inp["v"], inp["alpha"], inp["beta"], oa)
    gate = inp["alpha"][:, :, None].expand(-1, -1, w.d_k).contiguous()
    pb.step_kda(ids, inp["q"], inp["k"], inp["v"], gate, inp["beta"], ob)
    shape = (w.batch, w.n_v_heads, w.d_k, w.d_v)
    ca, cb = torch.empty(shape, dtype=torch.int8, device=DEV), torch.empty(shape, dtype=torch.int8, device=DEV)
    r = torch.empty((w.batch, w.n_v_heads, w.d_k), device=DEV)
    c = torch.empty((w.batch, w.n_v_heads, w.d_v), device=DEV)
    pa.export(ids, ca, r, c)
    pb.export(ids, cb, r, c)
    torch.cuda.synchronize()
    d = (ca.to(torch.int16) - cb.to(torch.int16)).abs()
    assert int(d.max()) <= 1 and int((d != 0).sum()) <= PT.CODE_MISMATCH_FRAC * d.numel()
    PT.compare_out(ob.cpu().numpy(), oa.double().cpu().numpy(), "kda vs gdn o")


@pytest.mark.parametrize("case", range(5))
def test_kda_ragged_shapes(case):
    """The generic (non-uniform layout) kernels with channel-wise gates."""
    Hv, Hqk, dk, dv, n_slots, bits = _ragged_cases()[case]
    _say(f"ragged kda case {case}: Hv={Hv} Hqk={Hqk} dk={dk} dv={dv}")
    rng = np.random.default_rng(200 + case)
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
    dg = rng.uniform(0.5, 1.0, (B, Hv, dk)); be = rng.uniform(0, 1, (B, Hv))
    t32 = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(DEV)
    o = torch.empty((B, Hv, dv), dtype=torch.float32, device=DEV)
    pool.step_kda(ids, t32(q), t32(k), t32(v), t32(dg), t32(be), o)
    out = torch.empty((n_slots, Hv, dk, dv), dtype=torch.int8, device=DEV)
    pool.export(all_ids, out, torch.empty((n_slots, Hv, dk), device=DEV), torch.empty((n_slots, Hv, dv), device=DEV))
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    hq = np.arange(Hv) // (Hv // Hqk)
    f32 = lambda a: a.astype(np.float32).astype(np.float64)
    qq, kk = f32(q)[:, hq].reshape(-1, dk), f32(k)[:, hq].reshape(-1, dk)
    tiles = (sel[:, None] * Hv + np.arange(Hv)[None]).reshape(-1)
    new, o_ref, y = oracle.decode_step(codes[tiles], r[tiles], c[tiles], tb_all[tiles], qq, kk,
                                       f32(v).reshape(-1, dv), f32(dg).reshape(-1, dk), f32(be).reshape(-1),
                                       want_y=True)
    PT.compare_codes(got.reshape(-1, dk, dv)[tiles], new, y, f"ragged kda case {case}")
    PT.compare_out(o.cpu().numpy().reshape(-1, dv), o_ref)
    untouched = np.setdiff1d(np.arange(n_slots), sel)
    for s in untouched:
        assert np.array_equal(got[s], codes.reshape(n_slots, Hv, dk, dv)[s])


def test_kda_argument_errors_and_prepared_call():
    w = W.workload(0)
    pool = stepq.Pool(2, w.n_v_heads, w.n_qk_heads, w.d_k, w.d_v, row_bits(w), device=DEV)
    z = lambda *s, dt=torch.float32: torch.zeros(s, dtype=dt, device=DEV)
    ids = torch.tensor([0, 1], dtype=torch.int32, device=DEV)
    with pytest.raises(ValueError):          # a per-head gate is not a channel-wise gate
        pool.step_kda(ids, z(2, 4, 64), z(2, 4, 64), z(2, 4, 64), z(2, 4), z(2, 4), z(2, 4, 64))
    pool.step_kda(ids[:0], z(0, 4, 64), z(0, 4, 64), z(0, 4, 64), z(0, 4, 64), z(0, 4), z(0, 4, 64))
    bits = row_bits(w)
    pa = build_pool(w, device=DEV, bits=bits)
    pb = build_pool(w, device=DEV, bits=bits)
    ids = W.active_slots(w).to(DEV)
    inp = W.step_inputs(w, 0, 0, device=DEV)
    gate = W.kda_gates(w, 0, 0, device=DEV)
    oa = torch.empty((w.batch, w.n_v_heads, w.d_v), dtype=torch.float32, device=DEV)
    ob = torch.empty_like(oa)
    pa.step_kda(ids, inp["q"], inp["k"], inp["v"], gate, inp["beta"], oa)
    pb.prepare_step(ids, inp["q"], inp["k"], inp["v"], gate, inp["beta"], ob)()
    torch.cuda.synchronize()
    assert torch.equal(oa, ob) and torch.equal(pa.memory, pb.memory)
