"""GPU parity at the extremes of the decode step, lockstep against the fp64
oracle through the C ABI: every slot of the 2048-slot pool stepped in one
launch (65,536 workgroups), the degenerate gates of the update:
alpha = 0 (the state is replaced by the rank-one write beta k v^T),
beta = 0 (pure decay, X = alpha S), and channel-wise gates of exactly 0 or 1
(rows forgotten or kept whole); and the dynamic range of the matrix-core
products, whose row weights are split into binary16 hi + lo parts under a
power-of-two prescale per tile: weights spanning ~40 binades inside a tile,
whole tiles at 2^60 and 2^-60 (outside binary16's range without the
prescale), and heads whose keys or queries are all zero."""
import dataclasses

import numpy as np
import pytest
import torch

from paper_2609_38169_amd import workloads as W
import _parity as PT

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda", 0)


def _say(*a):
    print(*a, flush=True)


def test_every_slot_of_the_pool():
    """B = n_slots = 2048: all 65,536 tiles of the pool in one launch."""
    w = dataclasses.replace(W.workload(2), batch=2048)
    assert int(W.active_slots(w).numel()) == w.n_slots
    PT.lockstep_run(w, 2, np.array([0, 1, 1023, 1024, 2046, 2047]), DEV, say=_say)


def _set(key, fn):
    def mutate(inp):
        inp = dict(inp)
        inp[key] = fn(inp[key])
        return inp
    return mutate


@pytest.mark.parametrize("refit", [False, True, "row_absmax"])
def test_zero_gate_replaces_state(refit):
    """alpha = 0: X = beta k v^T, whatever the stored codes."""
    w = W.workload(1)
    PT.lockstep_run(w, 3, np.arange(0, w.batch, 7), DEV, mutate=_set("alpha", torch.zeros_like), refit=refit,
                    say=_say)


def test_zero_beta_decays():
    """beta = 0: X = alpha S, the codes shrink by alpha and nothing is written."""
    w = W.workload(1)
    PT.lockstep_run(w, 4, np.arange(0, w.batch, 7), DEV, mutate=_set("beta", torch.zeros_like), say=_say)


def test_kda_gates_zero_or_one():
    """Channel-wise gates d_i in {0, 1}: forgotten rows hold only the write,
    kept rows add it to the whole old row."""
    w = W.workload(2)

    def binary(d):
        return (d > d.median()).to(d.dtype)

    PT.lockstep_run(w, 3, np.array([0, 255, 511]), DEV, mutate=_set("alpha", binary), kda=True, say=_say)


def _row_scaled(seed, lo, hi):
    def f(S):
        rng = np.random.default_rng(seed)
        e = rng.integers(lo, hi + 1, size=S.shape[:3]).astype(np.float64)
        return S.astype(np.float64) * np.exp2(e)[..., None]
    return f


def _tile_exponents(n_rows, n_heads):
    """Tiles of the checked rows alternately at 2^60, 1 and 2^-60."""
    return np.array([60.0, 0.0, -60.0])[np.arange(n_rows * n_heads) % 3].reshape(n_rows, n_heads)


def _spread_keys(seed, lo, hi):
    """Key entries scaled by 2^e, e uniform in lo..hi (exact in bf16)."""
    def mutate(inp):
        inp = dict(inp)
        rng = np.random.default_rng(seed)
        e = torch.from_numpy(np.exp2(rng.integers(lo, hi + 1, size=tuple(inp["k"].shape))).astype(np.float32))
        inp["k"] = (inp["k"].float() * e.to(inp["k"].device)).to(inp["k"].dtype)
        return inp
    return mutate


@pytest.mark.parametrize("kda", [False, True])
def test_weights_span_40_binades(kda):
    """Rows scaled by 2^[-4, 4] and key entries by 2^[-16, 16]: the k weights
    of one tile span ~40 binades, beyond the 17 over which the binary16
    hi + lo split keeps full precision.  fp32 itself then loses the fixed
    tie window's accuracy on a few codes, so mismatches and o are judged
    against the step's fp32 forward error bounds."""
    w = W.workload(2)
    PT.lockstep_run(w, 3, np.array([0, 200, 511]), DEV, kda=kda, say=_say, state_map=_row_scaled(7, -4, 4),
                    mutate=_spread_keys(8, -16, 16), fp32_bounds=True)


@pytest.mark.parametrize("refit,kda", [(False, False), (True, False), ("row_absmax", False), (False, True)])
def test_tiles_at_extreme_magnitudes(refit, kda):
    """Tiles at 2^60, 1 and 2^-60, their values v scaled with them, so the
    step is exactly equivariant under the scaling (X, o and the refitted
    factors scale by the same power of two): the weights lie far outside
    binary16's range until the per-tile prescale brings them in.  The fixed
    absolute part of the o limit does not scale with the tile, so o is also
    allowed the step's fp32 forward error bound (which does)."""
    w = W.workload(2)
    rows = np.array([1, 300, 510])
    e = _tile_exponents(len(rows), w.n_v_heads)

    def scale_state(S):
        return S.astype(np.float64) * np.exp2(e)[:, :, None, None]

    def scale_v(inp):
        inp = dict(inp)
        v = inp["v"].clone()
        f = torch.from_numpy(np.exp2(e).astype(np.float32)).to(v.device)
        idx = torch.as_tensor(rows, dtype=torch.long, device=v.device)
        v[idx] = (v[idx].float() * f[:, :, None]).to(v.dtype)
        inp["v"] = v
        return inp

    PT.lockstep_run(w, 3, rows, DEV, refit=refit, kda=kda, say=_say, state_map=scale_state, mutate=scale_v,
                    fp32_bounds=True)


@pytest.mark.parametrize("idx", [2, 3])
def test_saturating_updates(idx):
    """v scaled by 64 (exact in bf16): the rank-one write drives a large share
    of the new codes past +-q_b in both directions, on every row width of the
    workload's mix (8/4 for pool_b512, 8/4/2 for pool_4bit), so the clamp of
    the requantization (the FMA clamp bit on (y - 1)/S, and for 8-bit fields
    the convert's saturation at 255) decides them; lockstep with the oracle,
    which clips in fp64."""
    w = W.workload(idx)
    ls = PT.lockstep_run(w, 2, np.array([0, 255, 511]), DEV, mutate=_set("v", lambda v: v * 64), say=_say)
    assert ls.saturated > 0.05, f"only {ls.saturated:.3f} of the checked codes saturated"


def test_zero_keys_and_queries():
    """All-zero k on some q/k heads and all-zero q on others: a tile whose
    largest k (or q) weight is 0.  With k = 0 the step is a pure decay,
    y = alpha q exactly; the gates are put on odd multiples of 2^-8 so that
    alpha q is never exactly half-way between codes (an exact tie, which the
    kernel rounds to even and the fp64 oracle's own rounding of
    X q_b / (r c) decides either way)."""
    w = W.workload(2)

    def zero_heads(inp):
        inp = dict(inp)
        k, q = inp["k"].clone(), inp["q"].clone()
        k[:, 0::3] = 0
        q[:, 1::3] = 0
        m = torch.round(inp["alpha"].float() * 256.0)
        m = m - (1 - torch.remainder(m, 2))          # the odd multiple of 2^-8 at or below
        inp["k"], inp["q"], inp["alpha"] = k, q, (m / 256.0).to(inp["alpha"].dtype)
        return inp

    PT.lockstep_run(w, 3, np.array([2, 256, 509]), DEV, mutate=zero_heads, say=_say)


@pytest.mark.parametrize("idx,refit", [(1, False), (1, True), (2, False), (2, "row_absmax")])
def test_adjacent_slots_hint_changes_nothing(idx, refit):
    """STEPQ_STEP_ADJACENT_SLOTS only reorders the tiles of a launch: codes,
    scales and o are bit-identical with and without it, on a batch of
    adjacent slots (layer_b64) and on a scattered one (pool_b512), where the
    hint is wrong."""
    from paper_2609_38169_amd.pools import build_pool
    from paper_2609_38169_amd import stepq
    w = W.workload(idx)
    slots = W.active_slots(w).to(DEV)
    _say(f"adjacent hint {w.name} refit={refit}: building two pools")
    pools = [build_pool(w, 0, device=DEV) for _ in range(2)]
    outs = []
    for adjacent, pool in zip((False, True), pools):
        o = torch.empty((w.batch, w.n_v_heads, w.d_v), dtype=torch.float32, device=DEV)
        for t in range(2):
            inp = W.step_inputs(w, 0, t, device=DEV)
            pool.step(slots, inp["q"], inp["k"], inp["v"], inp["alpha"], inp["beta"], o, refit=refit,
                      adjacent=adjacent)
        n = w.batch
        codes = torch.empty((n, w.n_v_heads, w.d_k, w.d_v), dtype=torch.int8, device=DEV)
        r = torch.empty((n, w.n_v_heads, w.d_k), dtype=torch.float32, device=DEV)
        c = torch.empty((n, w.n_v_heads, w.d_v), dtype=torch.float32, device=DEV)
        pool.export(slots, codes, r, c)
        torch.cuda.synchronize()
        outs.append((codes.cpu(), r.cpu(), c.cpu(), o.cpu()))
    for a, b in zip(*outs):
        assert torch.equal(a.view(torch.uint8) if a.dtype == torch.int8 else a.view(torch.int32),
                           b.view(torch.uint8) if b.dtype == torch.int8 else b.view(torch.int32))
    _say(f"adjacent hint {w.name}: bit-identical")


def test_stream_ref_moves_memory_only():
    """The memory-only reference of a decode launch (a measurement aid)
    leaves every byte of the pool as it was and writes zeros to o, on a
    uniform pool (pool_b512) and on a pool with a head list (layer_b64's
    two layout classes); it takes the adjacent-slots hint only."""
    import ctypes
    from paper_2609_38169_amd import stepq
    from paper_2609_38169_amd.pools import build_pool, row_bits
    for idx in (2, 1):
        w = W.workload(idx)
        pool = build_pool(w, device=DEV, bits=row_bits(w))
        before = pool.memory.clone()
        ids = W.active_slots(w).to(DEV)
        inp = W.step_inputs(w, 0, 0, device=DEV)
        o = torch.full((w.batch, w.n_v_heads, w.d_v), 7.0, dtype=torch.float32, device=DEV)
        pool.prepare_stream_ref(ids, inp["q"], inp["k"], inp["v"], inp["alpha"], inp["beta"], o)()
        torch.cuda.synchronize()
        assert torch.equal(before, pool.memory), w.name
        assert torch.count_nonzero(o).item() == 0, w.name
    a = stepq._step_args(pool, ids, inp["q"], inp["k"], inp["v"], inp["alpha"], inp["beta"], o, None, False)
    with pytest.raises(stepq.StepqError):
        stepq._check(stepq.lib().stepq_decode_stream_ref(*a[:9], ctypes.c_uint32(stepq.STEPQ_STEP_REFIT), *a[9:]))
