"""CPU-side checks of the product library: it loads and exports every
declared entry point, its layout sizes and its setup step agree with the
oracle's independent versions, and bad descriptors are rejected without a
device."""
import ctypes
import os
import re

import numpy as np
import pytest
import torch

import oracle
from paper_2609_38169_amd import stepq, workloads as W
from paper_2609_38169_amd.pools import row_bits

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_library_exports_every_declared_symbol():
    text = open(os.path.join(ROOT, "include", "stepq.h")).read()
    declared = set(re.findall(r"^\s*(?:[\w\s\*]+?)\b(stepq_\w+)\s*\(", text, re.M))
    assert {"stepq_pool_create", "stepq_decode_step", "stepq_pool_dequant"} <= declared
    L = stepq.lib()
    for name in sorted(declared):
        assert hasattr(L, name), name
    assert declared == set(stepq.EXPORTED)


@pytest.mark.parametrize("idx", [0, 1, 2, 3, 4])
def test_pool_bytes_match_oracle_layout(idx):
    w = W.workload(idx)
    bits = W.bit_map_draw(w).numpy() if w.bits != "lifetime48" else stepq.stepq_setup_lifetime_bits(
        W.calibration_gates(w), w.d_k)
    pb, sb = stepq.stepq_pool_bytes(w.n_slots, w.n_v_heads, w.n_qk_heads, w.d_k, w.d_v, bits)
    assert sb == oracle.slot_bytes(bits, w.d_v)
    assert pb == sb * w.n_slots
    if idx in (2, 4):
        assert sb == w.n_v_heads * 13312
    if idx == 4:       # 48 layers x 256 slots: 4.875 GiB vs 24 GiB of fp32 states
        assert w.layers * pb == 4.875 * 2 ** 30
        assert w.layers * w.n_slots * w.n_v_heads * w.d_k * w.d_v * 4 == 24 * 2 ** 30


def test_pivot_heads_padded_to_a_uniform_mix():
    """Integer rows that fit a uniform mix are stored in it, width classes
    padded with empty groups: a 6-bit head with 2 pivot rows keeps the
    12,288-byte codes region of 64 @ 8 + 64 @ 4 (tight it would be 94
    groups); rows that fit no mix stay tight.  Library and oracle agree."""
    def head(n16, n8, n4, n2):
        b = np.array([16] * n16 + [8] * n8 + [4] * n4 + [2] * n2, np.uint8)
        return np.random.default_rng(n16 + 3 * n8).permutation(b)

    cases = [
        (head(2, 62, 64, 0), 12288 + 2 * 256 + 1024),             # {8,4,0}: 2 empty 8-bit groups
        (head(3, 64, 61, 0), 12288 + 3 * 256 + 1024),             # one 4-bit group half empty, one empty
        (head(8, 30, 30, 60), 8192 + 8 * 256 + 1024),             # {4,2,2}
        (head(5, 123, 0, 0), 16384 + 5 * 256 + 1024),             # {16,0,0}
        (head(32, 0, 0, 96), 4096 + 32 * 256 + 1024),             # {0,0,4} with the most pivot rows
        (head(8, 100, 20, 0), (100 + 10) * 128 + 8 * 256 + 1024),  # fits no mix: tight
        (head(0, 64, 64, 0), 13312),                              # no pivots: the uniform layout itself
    ]
    for bits, tile in cases:
        bits = bits[None]
        pb, sb = stepq.stepq_pool_bytes(2, 1, 1, 128, 128, bits)
        assert sb == tile, (sb, tile)
        assert oracle.slot_bytes(bits, 128) == tile
    # the padded groups hold only zero bytes in the oracle's own packing
    bits = head(2, 62, 64, 0)[None]
    rng = np.random.default_rng(5)
    codes = rng.integers(-7, 8, size=(1, 1, 128, 128)).astype(np.int8)
    img = oracle.pack_pool(codes, np.ones((1, 1, 128), np.float32), np.ones((1, 1, 128), np.float32), bits,
                           pv=np.zeros((1, 1, 128, 128), np.uint16))
    assert not img[62 * 128:64 * 128].any()                       # 8-bit groups 62, 63 are empty
    assert img[64 * 128:96 * 128].any()                           # the 4-bit groups follow at group 64


def test_ragged_layout_sizes():
    rng = np.random.default_rng(0)
    for dk, dv in [(37, 64), (96, 128), (1, 64), (128, 128)]:
        bits = rng.choice([2, 4, 8], size=(5, dk)).astype(np.uint8)
        pb, sb = stepq.stepq_pool_bytes(3, 5, 5, dk, dv, bits)
        assert sb == oracle.slot_bytes(bits, dv) and pb == 3 * sb
        bits[rng.random(bits.shape) < 0.1] = 16          # FP16 pivot rows
        pb, sb = stepq.stepq_pool_bytes(3, 5, 5, dk, dv, bits)
        assert sb == oracle.slot_bytes(bits, dv) and pb == 3 * sb


def test_whole_fp16_head_layout():
    """A 128x128 head whose every row is an FP16 pivot is accepted (the
    paper's Qwen pivots are whole heads): its tile is 32 KiB of binary16
    values plus the unused r and c slots, as the oracle's packer lays it out.
    Between 33 and 127 pivot rows a head is refused."""
    rng = np.random.default_rng(3)
    bits = rng.permutation(np.repeat(np.array([8, 4], np.uint8), 64))[None].repeat(4, 0)
    bits[1] = 16
    bits[3] = 16
    pb, sb = stepq.stepq_pool_bytes(2, 4, 4, 128, 128, bits)
    assert sb == oracle.slot_bytes(bits, 128) == 2 * 13312 + 2 * (128 * 256 + 1024)
    for n16, status in [(32, None), (33, 2), (127, 2)]:
        b = bits.copy()
        b[1] = 8
        b[1, :n16] = 16
        if status is None:
            assert stepq.stepq_pool_bytes(2, 4, 4, 128, 128, b)[1] == oracle.slot_bytes(b, 128)
        else:
            with pytest.raises(stepq.StepqError) as e:
                stepq.stepq_pool_bytes(2, 4, 4, 128, 128, b)
            assert e.value.status == status
    with pytest.raises(stepq.StepqError) as e:           # whole FP16 heads need d_k = d_v = 128
        stepq.stepq_pool_bytes(2, 4, 4, 128, 64, bits)
    assert e.value.status == 2


@pytest.mark.parametrize("bad,status", [
    (dict(n_slots=0), 1), (dict(n_v_heads=6, n_qk_heads=4), 1), (dict(d_k=129), 2), (dict(d_v=96), 2),
    (dict(bitval=3), 1), (dict(bitval=12), 1),
    (dict(bitval=16), 2),                       # 64 pivot rows per 64x64 head: more than the 32 supported
    # 130,000 whole FP16 128x128 heads: a 4.4 GB slot record, past the 32-bit tile offsets
    (dict(n_v_heads=130000, n_qk_heads=1, d_k=128, d_v=128, bitval=16), 2),
])
def test_bad_descriptor_rejected(bad, status):
    a = dict(n_slots=2, n_v_heads=4, n_qk_heads=2, d_k=64, d_v=64)
    bitval = bad.pop("bitval", 8)
    a.update(bad)
    bits = np.full((a["n_v_heads"], a["d_k"]), bitval, np.uint8)
    with pytest.raises(stepq.StepqError) as e:
        stepq.stepq_pool_bytes(a["n_slots"], a["n_v_heads"], a["n_qk_heads"], a["d_k"], a["d_v"], bits)
    assert e.value.status == status


def test_null_descriptor_rejected():
    L = stepq.lib()
    assert L.stepq_pool_bytes(None, None, None) == 1
    out = ctypes.c_void_p()
    assert L.stepq_pool_create(None, None, 0, ctypes.byref(out)) == 1
    assert L.stepq_decode_step(None, None, 0, None, None, None, None, None, 0, None, None) == 1


@pytest.mark.parametrize("idx", [0, 1, 3])
def test_setup_fit_matches_oracle(idx):
    """The library's host fit and the oracle's are written separately; both
    evaluate the same double-precision formulas, so the fp32 scales agree
    bit for bit."""
    w = W.workload(idx)
    slots = range(0, min(4, w.n_slots))
    S = W.initial_state(w, 0, slots).numpy()
    r1, c1 = stepq.stepq_setup_fit(S, n_threads=3)
    r2, c2 = oracle.fit_absmax(S.reshape(-1, w.d_k, w.d_v))
    assert np.array_equal(r1.reshape(r2.shape), r2)
    assert np.array_equal(c1.reshape(c2.shape), c2)
    wts = np.random.default_rng(1).uniform(0.5, 2, S.shape[:-1]).astype(np.float32)
    r1, c1 = stepq.stepq_setup_fit(S, wts)
    r2, c2 = oracle.fit_absmax(S.reshape(-1, w.d_k, w.d_v), wts.reshape(-1, w.d_k).astype(np.float64))
    assert np.array_equal(r1.reshape(r2.shape), r2) and np.array_equal(c1.reshape(c2.shape), c2)
    # pivot rows (16) left out of the column factors
    bits = np.random.default_rng(2).choice([4, 8, 16], size=S.shape[:-1], p=[0.45, 0.45, 0.1]).astype(np.uint8)
    r1, c1 = stepq.stepq_setup_fit(S, wts, row_bits=bits)
    r2, c2 = oracle.fit_absmax(S.reshape(-1, w.d_k, w.d_v), wts.reshape(-1, w.d_k).astype(np.float64),
                               bits=bits.reshape(-1, w.d_k))
    assert np.array_equal(r1.reshape(r2.shape), r2) and np.array_equal(c1.reshape(c2.shape), c2)
    # the N2 level normalisation (top level 2^(8-b) q_b per width)
    bits = np.random.default_rng(3).choice([2, 4, 8, 16], size=S.shape[:-1]).astype(np.uint8)
    r1, c1 = stepq.stepq_setup_fit(S, wts, row_bits=bits, levels=stepq.STEPQ_LEVELS_POW2, n_threads=2)
    r2, c2 = oracle.fit_absmax(S.reshape(-1, w.d_k, w.d_v), wts.reshape(-1, w.d_k).astype(np.float64),
                               bits=bits.reshape(-1, w.d_k), levels=oracle.LEVELS_POW2)
    assert np.array_equal(r1.reshape(r2.shape), r2) and np.array_equal(c1.reshape(c2.shape), c2)
    with pytest.raises(ValueError):
        stepq.stepq_setup_fit(S, levels=stepq.STEPQ_LEVELS_POW2)
    with pytest.raises(stepq.StepqError):
        stepq.stepq_pool_bytes(2, 4, 4, 16, 64, np.full((4, 16), 8, np.uint8), levels=7)


@pytest.mark.parametrize("levels", [0, 1])
def test_setup_fit_meets_its_definition(levels):
    """The library's setup fit against Section 4.3's definitions directly,
    not through the oracle: r_i is the fp32 rounding of (m_i / w_i)^(1/2),
    m_i = mean_j |S_ij|; every integer entry lies within its row and column
    factors, r_i c_j top_i >= |S_ij| (top_i = 1 under N1, 2^(8-b) q_b under
    N2); each column's factor is the smallest fp32 value with that property
    (the column's largest entry reaches the top level); pivot rows take no
    part in the column factors; all-zero rows and columns get the floor
    2^-60."""
    rng = np.random.default_rng(31)
    n, dk, dv = 6, 40, 64
    S = (rng.standard_normal((n, dk, dv)) * np.exp(rng.standard_normal((n, dk, 1)))).astype(np.float32)
    S[1, 3, :] = 0.0                      # a zero row
    S[2, :, 5] = 0.0                      # a zero column
    wts = np.exp(0.5 * rng.standard_normal((n, dk))).astype(np.float32)
    bits = rng.choice([2, 4, 8, 16], size=(n, dk), p=[0.3, 0.3, 0.3, 0.1]).astype(np.uint8)
    bits[2, :] = np.where(bits[2, :] == 16, 8, bits[2, :])
    r, c = stepq.stepq_setup_fit(S, wts, row_bits=bits, levels=levels)
    floor = 2.0 ** -60
    m = np.abs(S.astype(np.float64)).mean(axis=2)
    r_def = np.maximum(np.sqrt(m / wts.astype(np.float64)), floor)
    assert np.all(np.abs(r.astype(np.float64) - r_def) <= np.spacing(r_def.astype(np.float32)).astype(np.float64)), \
        "r is not the fp32 rounding of (m / w)^(1/2)"
    assert r[1, 3] == np.float32(floor)
    b = bits.astype(np.int64)
    qb = 2.0 ** (b - 1) - 1
    top = qb * 2.0 ** (8 - b) if levels else np.ones_like(qb)
    ints = (bits != 16)[:, :, None]
    bound = r.astype(np.float64)[:, :, None] * c.astype(np.float64)[:, None, :] * top[:, :, None]
    assert np.all(np.where(ints, bound >= np.abs(S.astype(np.float64)), True)), "an entry exceeds r c top"
    need = np.where(ints, np.abs(S.astype(np.float64)) / (r.astype(np.float64) * top)[:, :, None], 0.0).max(axis=1)
    need = np.maximum(need, floor)
    c64 = c.astype(np.float64)
    assert np.all(c64 >= need)
    below = np.nextafter(c, np.float32(0)).astype(np.float64)
    assert np.all((below < need) | (c == np.float32(floor))), "a column factor is larger than it needs to be"
    assert c[2, 5] == np.float32(floor)
    # pivot rows do not move the column factors: scaling them changes nothing
    S2 = S.copy()
    S2[bits == 16] *= 1000.0
    _, c2 = stepq.stepq_setup_fit(S2, wts, row_bits=bits, levels=levels)
    assert np.array_equal(c, c2)


def test_lifetime_bits_match_oracle():
    w = W.workload(1)
    g = W.calibration_gates(w)
    b1 = stepq.stepq_setup_lifetime_bits(g, w.d_k, 6.0, 4, 8)
    b2 = oracle.lifetime_bitmap(g.numpy(), w.d_k, 6.0, 4, 8)
    assert np.array_equal(b1, b2)
    assert b1.astype(float).mean() == 6.0
    # {2,4}/{4,8} with other budgets
    for bud, lo, hi in [(5.0, 4, 8), (3.0, 2, 4), (8.0, 4, 8), (4.0, 4, 8)]:
        assert np.array_equal(stepq.stepq_setup_lifetime_bits(g, 16, bud, lo, hi),
                              oracle.lifetime_bitmap(g.numpy(), 16, bud, lo, hi))
    with pytest.raises(stepq.StepqError):
        stepq.stepq_setup_lifetime_bits(g, 16, 9.0, 4, 8)


def test_workload_draws_are_seeded():
    w = W.workload(0)
    a = W.step_inputs(w, 0, 3)
    b = W.step_inputs(w, 0, 3)
    for key in a:
        assert torch.equal(a[key], b[key])
    assert not torch.equal(a["q"], W.step_inputs(w, 0, 4)["q"])
    qn = torch.linalg.vector_norm(a["q"].double(), dim=-1)
    assert torch.allclose(qn, torch.ones_like(qn), atol=1e-6)
    S = W.initial_state(w)
    assert abs(float(S.std()) - 0.05) < 0.005
    s2 = W.initial_state(W.workload(2), 0, range(5, 6))
    assert torch.equal(s2, W.initial_state(W.workload(2), 0, range(5, 7))[:1])
    assert sorted(torch.cat(W.rotation_slots(W.workload(2))).tolist()) == list(range(2048))
    bits = W.bit_map_draw(W.workload(3)).numpy()
    assert all(sorted(np.bincount(row, minlength=9)[[2, 4, 8]]) == [32, 32, 64] for row in bits)
    for idx in range(5):                     # channel-wise gates: shape, dtype, range, seeded, own stream
        wk = W.workload(idx)
        d = W.kda_gates(wk, 0, 1)
        assert d.shape == (wk.batch, wk.n_v_heads, wk.d_k) and d.dtype == wk.act_dtype
        assert torch.equal(d, W.kda_gates(wk, 0, 1)) and not torch.equal(d, W.kda_gates(wk, 0, 2))
        assert float(d.min()) > 0.0 and float(d.max()) <= 1.0


def test_library_device_code_is_gfx950():
    """The library must carry device code for gfx950 and nothing else (a
    mixed hipcc command line once silently fell back to another target)."""
    from paper_2609_38169_amd.build import device_targets
    assert device_targets(stepq.LIB_PATH) == ["gfx950"]


# ---------------------------------------------------------------- calibration side (host code vs oracle)
def _calib_stream(seed, T=30, H=3, dk=8, kda=True):
    rng = np.random.default_rng(seed)
    q = rng.standard_normal((T, H, dk)).astype(np.float32)
    k = rng.standard_normal((T, H, dk)).astype(np.float32)
    q /= np.linalg.norm(q, axis=-1, keepdims=True)
    k /= np.linalg.norm(k, axis=-1, keepdims=True)
    beta = rng.uniform(0, 1, (T, H)).astype(np.float32)
    gate = (rng.uniform(0.7, 1.0, (T, H, dk)) if kda else rng.uniform(0.7, 1.0, (T, H))).astype(np.float32)
    return q, k, beta, gate


@pytest.mark.parametrize("kda", [False, True])
def test_row_impact_matches_oracle(kda):
    import oracle.calibration as CAL
    q, k, beta, gate = _calib_stream(10, kda=kda)
    w, om = stepq.stepq_setup_row_impact(q, k, beta, gate)
    w_o, om_o = CAL.row_impact(q, k, beta, gate)
    np.testing.assert_allclose(om, om_o, rtol=1e-12)
    np.testing.assert_allclose(w, w_o, rtol=2e-7)


@pytest.mark.parametrize("unit", ["row", "head"])
def test_distortion_matches_oracle(unit):
    import oracle.calibration as CAL
    rng = np.random.default_rng(11)
    C, H, dk, dv = 3, 2, 12, 16
    S = (rng.standard_normal((C, H, dk, dv)) * np.exp(rng.standard_normal((C, H, dk, 1)))).astype(np.float32)
    w = np.exp(0.3 * rng.standard_normal((H, dk))).astype(np.float32)
    piv = np.zeros((H, dk), bool)
    piv[1, 4] = True
    for pv in (None, piv):
        d = stepq.stepq_setup_distortion(S, [2, 4, 8, 16], unit, row_weight=w, pivots=pv, n_threads=3)
        d_o = CAL.calib_distortion(S.astype(np.float64), [2, 4, 8, 16], unit, w=w.astype(np.float64), pivots=pv)
        np.testing.assert_allclose(d, d_o, rtol=1e-12)


def test_lifetime_weights_and_pivots_match_oracle():
    import oracle.calibration as CAL
    ell = np.array([-0.5, -0.02, -1e-6, 0.0, -3e-13])
    np.testing.assert_allclose(stepq.stepq_setup_lifetime_weights(ell, 512), CAL.lifetime_weights(ell, 512),
                               rtol=1e-9)
    risk = np.random.default_rng(12).uniform(0, 1, 40)
    assert np.array_equal(stepq.stepq_setup_select_pivots(risk, 5), CAL.select_pivots(risk, 5))


@pytest.mark.parametrize("kda", [False, True])
def test_mean_log_retention_and_costs_match_oracle(kda):
    """ell per key row and per head, the lifetime-weighted costs and the
    pivot risk from libstepq against the oracle's loops; constant gates give
    log g exactly (Appendix A.3)."""
    import oracle.calibration as CAL
    rng = np.random.default_rng(14)
    T, H, dk = 9, 3, 7
    g = rng.uniform(0.5, 1.0, (T, H, dk) if kda else (T, H)).astype(np.float32)
    for unit in ("row", "head"):
        np.testing.assert_allclose(stepq.stepq_setup_mean_log_retention(g, dk, unit),
                                   CAL.mean_log_retention_units(g, dk, unit), rtol=1e-12, atol=1e-15)
    const = np.full(g.shape, 0.75, np.float32)
    np.testing.assert_allclose(stepq.stepq_setup_mean_log_retention(const, dk, "head"), np.log(0.75), rtol=1e-12)
    L = rng.uniform(1, 50, H * dk)
    d = rng.uniform(0, 1, (H * dk, 4))
    np.testing.assert_allclose(stepq.stepq_setup_lifetime_costs(L, d, 3), L[:, None] * d[:, :3], rtol=1e-15)
    np.testing.assert_allclose(stepq.stepq_setup_pivot_risk(L, d, 2, 3), L * (d[:, 2] - d[:, 3]), rtol=1e-15)
    with pytest.raises(stepq.StepqError):
        stepq.stepq_setup_mean_log_retention(np.zeros((2, H), np.float32), dk, "row")


def test_allocators_match_oracle():
    import oracle.calibration as CAL
    rng = np.random.default_rng(13)
    cands = [2, 4, 8]
    for trial in range(25):
        U = int(rng.integers(2, 12))
        n_u = rng.choice([64, 128], size=U).astype(np.int32)
        cost = np.sort(rng.uniform(0, 1, (U, 3)), axis=1)[:, ::-1] * rng.uniform(0.1, 10, (U, 1))
        budget = float(rng.choice([2.5, 3.0, 4.0, 5.0, 6.0, 7.9]))
        dp = stepq.stepq_setup_allocate(cost, n_u, cands, budget, "dp")
        dp_o = CAL.allocate_dp(cost, n_u, cands, budget)
        tot = lambda ch: sum(cost[u, ch[u]] for u in range(U))
        assert abs(tot(dp) - tot(dp_o)) <= 1e-12 * max(1.0, tot(dp_o))
        lg = stepq.stepq_setup_allocate(cost, n_u, cands, budget, "lagrangian")
        lg_o = CAL.allocate_lagrangian(cost, n_u, cands, budget)
        assert np.array_equal(lg, lg_o)
    with pytest.raises(stepq.StepqError):        # nothing fits
        stepq.stepq_setup_allocate(np.ones((3, 3)), 64, cands, 1.0, "dp")


@pytest.mark.parametrize("unit,kda", [("row", True), ("head", False)])
def test_calibration_pipeline_meets_the_budget(unit, kda):
    """calibrate(): pivots are the requested count, the integer units meet the
    average budget, and wider codes go to units whose lifetime-weighted
    distortion gains most."""
    from paper_2609_38169_amd.calibrate import calibrate
    q, k, beta, gate = _calib_stream(14, T=40, H=4, dk=16, kda=kda)
    rng = np.random.default_rng(15)
    S = (rng.standard_normal((6, 4, 16, 64)) * 0.1).astype(np.float32)
    cal = calibrate(q, k, beta, gate, S, budget=5.0, cand_bits=(2, 4, 8), unit=unit,
                    n_pivots=3 if unit == "row" else 1, horizon=256)
    bits = cal.row_bits
    piv = bits == 16
    units_piv = piv.sum() if unit == "row" else piv.all(axis=1).sum()
    assert units_piv == (3 if unit == "row" else 1)
    integer = bits[~piv].astype(np.float64)
    assert integer.mean() <= 5.0 + 1e-9 and set(np.unique(integer)) <= {2, 4, 8}
    np.testing.assert_allclose(np.exp(np.log(cal.row_weight.astype(np.float64)).mean(axis=1)), 1.0, rtol=1e-6)
    pb, sb = stepq.stepq_pool_bytes(2, 4, 4, 16, 64, bits)        # a valid pool layout
    assert pb == 2 * sb


def test_synthetic_pivot_draws():
    """The seeded pivot draws are reproducible and have the stated shape:
    1-3 pivot rows in a share of the heads, or whole FP16 heads."""
    w = W.workload(2)
    m = W.pivot_mask_draw(w)
    assert m.shape == (w.n_v_heads, w.d_k) and torch.equal(m, W.pivot_mask_draw(w))
    per_head = m.sum(1)
    assert per_head.max() <= 3 and 0 < (per_head > 0).sum() < w.n_v_heads
    for count in (1, 2, 5):
        h = W.pivot_head_draw(w, 0, count)
        assert h.shape == (w.n_v_heads,) and int(h.sum()) == count and torch.equal(h, W.pivot_head_draw(w, 0, count))
    assert not torch.equal(W.pivot_head_draw(w, 0, 2), W.pivot_head_draw(w, 1, 2))


def _plan_cases():
    """Descriptors of every planning path: each workload's map, uniform mixes
    side by side, padded pivot heads, whole FP16 heads, row-mix heads,
    generic heads, d_v = 64 and ragged d_k."""
    rng = np.random.default_rng(21)
    cases = []
    for i in range(5):
        w = W.workload(i)
        cases.append((w.name, w.n_v_heads, w.n_qk_heads, w.d_k, w.d_v, row_bits(w)))

    def mix(m8, m4, m2, piv=0):
        b = np.array([8] * m8 + [4] * m4 + [2] * m2, np.uint8)
        b[rng.choice(128, piv, replace=False)] = 16
        return rng.permutation(b)
    heads = [mix(64, 64, 0), mix(128, 0, 0), mix(0, 128, 0), mix(64, 64, 0, 3), np.full(128, 16, np.uint8)]
    cases.append(("compiled classes", 5, 5, 128, 128, np.stack(heads)))
    cases.append(("rowmix", 6, 3, 128, 128, np.stack([mix(n8, 128 - n8, 0, p) for n8, p in
                                                      [(50, 0), (70, 3), (61, 8), (88, 1), (40, 2), (99, 0)]])))
    cases.append(("generic + uniform", 4, 2, 128, 128,
                  np.stack([mix(64, 64, 0), rng.choice([2, 4, 8], 128).astype(np.uint8), mix(64, 64, 0),
                            mix(30, 50, 48)])))
    cases.append(("d_v 64", 3, 1, 37, 64, rng.choice([2, 4, 8, 16], (3, 37), p=[.3, .3, .3, .1]).astype(np.uint8)))
    cases.append(("ragged d_k", 2, 2, 96, 128, rng.choice([2, 4, 8], (2, 96)).astype(np.uint8)))
    return cases


@pytest.mark.parametrize("flags", [0, stepq.STEPQ_STEP_REFIT, stepq.STEPQ_STEP_ROW_ABSMAX])
def test_pool_plan_launches_cover_every_head_once(flags):
    """stepq_pool_plan (host only): the launches of a decode step cut the
    head order into consecutive slices that cover it, and the head order is
    a permutation of the value heads; the library's own plan check (the one
    stepq_pool_create runs) accepts every case."""
    for name, Hv, Hqk, dk, dv, bits in _plan_cases():
        launches, order = stepq.stepq_pool_plan(2, Hv, Hqk, dk, dv, bits, flags=flags)
        assert sorted(order.tolist()) == list(range(Hv)), name
        pos = 0
        for body, first, n in launches:
            assert first == pos and n >= 1, (name, launches)
            pos += n
        assert pos == Hv, (name, launches)


def test_pool_plan_launch_counts():
    """One launch for the uniform workloads, one combined launch for
    layer_b64's two classes of whole 8- and 4-bit heads when frozen, one per
    class when refitting."""
    for i in (0, 2, 3, 4):
        w = W.workload(i)
        assert len(stepq.stepq_pool_plan(1, w.n_v_heads, w.n_qk_heads, w.d_k, w.d_v, row_bits(w))[0]) == 1
    w = W.workload(1)
    assert len(stepq.stepq_pool_plan(1, w.n_v_heads, w.n_qk_heads, w.d_k, w.d_v, row_bits(w))[0]) == 1
    refit = stepq.stepq_pool_plan(1, w.n_v_heads, w.n_qk_heads, w.d_k, w.d_v, row_bits(w),
                                  flags=stepq.STEPQ_STEP_REFIT)[0]
    assert len(refit) == 2 and sum(n for _, _, n in refit) == w.n_v_heads
    with pytest.raises(stepq.StepqError):
        stepq.stepq_pool_plan(1, 2, 1, 128, 128, np.full((2, 128), 6, np.uint8))
