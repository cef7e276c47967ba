"""Pins for the fp64 oracle against what the paper and the mathematics fix.

Each test targets a mistake the oracle could plausibly contain (a dropped
term, a wrong sign, a transposed operand, a wrong level set or tie rule)
and checks it against something other than the oracle itself: a closed
form, an identity the paper proves, a different algebraic form of the same
equation, brute-force enumeration, or an integer the paper prints.
"""
import itertools
import json
import math
import os

import numpy as np
import pytest

import oracle

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_accounting.json")))


def _unit(rng, n, d):
    x = rng.standard_normal((n, d))
    return x / np.linalg.norm(x, axis=1, keepdims=True)


def _case(seed=0, n=3, dk=16, dv=12):
    rng = np.random.default_rng(seed)
    S = rng.standard_normal((n, dk, dv)) * 0.3
    q, k = _unit(rng, n, dk), _unit(rng, n, dk)
    v = rng.standard_normal((n, dv))
    alpha = rng.uniform(0.5, 1.0, n)
    beta = rng.uniform(0.0, 1.0, n)
    return rng, S, q, k, v, alpha, beta


# ---------------------------------------------------------------- update (Eq. 1, 2, 4)
def test_update_matches_affine_form():
    """Eq. 1 (first form, in the oracle) equals the affine form of Eq. 2,
    S_t = A S + B with A = (I - beta k k^T) alpha, B = beta k v^T, written
    here independently; the readout is y = X^T q (Eq. 4)."""
    _, S, q, k, v, alpha, beta = _case()
    X, o = oracle.update_fp(S, q, k, v, alpha, beta)
    for t in range(S.shape[0]):
        dk = S.shape[1]
        A = (np.eye(dk) - beta[t] * np.outer(k[t], k[t])) * alpha[t]
        Bm = beta[t] * np.outer(k[t], v[t])
        Xr = A @ S[t] + Bm
        np.testing.assert_allclose(X[t], Xr, rtol=0, atol=1e-13)
        np.testing.assert_allclose(o[t], Xr.T @ q[t], rtol=0, atol=1e-13)


def test_identity_gate_zero_write():
    """alpha = 1, beta = 0: the state is unchanged exactly and o = S^T q."""
    _, S, q, k, v, _, _ = _case(1)
    n = S.shape[0]
    X, o = oracle.update_fp(S, q, k, v, np.ones(n), np.zeros(n))
    assert np.array_equal(X, S)
    for t in range(n):
        np.testing.assert_allclose(o[t], S[t].T @ q[t], rtol=0, atol=1e-14)


def test_full_write_recalls_value():
    """alpha = 1, beta = 1, |k| = 1: the retrieval of the new state along k is
    the written value, X^T k = v (the Delta rule's defining property)."""
    _, S, q, k, v, _, _ = _case(2)
    n = S.shape[0]
    X, o = oracle.update_fp(S, q, k, v, np.ones(n), np.ones(n))
    for t in range(n):
        np.testing.assert_allclose(X[t].T @ k[t], v[t], rtol=0, atol=1e-12)
    # reading with q := k returns v as well
    X2, o2 = oracle.update_fp(S, k, k, v, np.ones(n), np.ones(n))
    np.testing.assert_allclose(o2, v, rtol=0, atol=1e-12)


def test_directional_contraction_identity():
    """Appendix B.1, Eq. self_correction:
    ||alpha (I - beta k k^T) E||_F^2 = alpha^2 [ ||E||^2 - beta (2 - beta |k|^2) ||k^T E||^2 ].
    With v = 0 the oracle's update maps E to alpha (I - beta k k^T) E."""
    rng = np.random.default_rng(3)
    n, dk, dv = 4, 10, 7
    E = rng.standard_normal((n, dk, dv))
    k = rng.standard_normal((n, dk)) * 0.4        # not unit: exercises the |k|^2 term
    q = rng.standard_normal((n, dk))
    alpha = rng.uniform(0.2, 1.0, n)
    beta = rng.uniform(0.0, 1.0, n)
    X, _ = oracle.update_fp(E, q, k, np.zeros((n, dv)), alpha, beta)
    for t in range(n):
        lhs = np.sum(X[t] ** 2)
        kE = k[t] @ E[t]
        rhs = alpha[t] ** 2 * (np.sum(E[t] ** 2) - beta[t] * (2 - beta[t] * k[t] @ k[t]) * kE @ kE)
        assert lhs == pytest.approx(rhs, rel=1e-12)


def test_row_readout_sensitivity():
    """Appendix B.3 / Eq. kda_sensitivity with d_i = alpha: a unit-norm error
    confined to key row i is read at the next step with squared norm g_i^2,
    g = A^T q = alpha (q - beta k (k^T q))."""
    rng = np.random.default_rng(4)
    dk, dv = 9, 6
    q, k = _unit(rng, 1, dk)[0], _unit(rng, 1, dk)[0]
    alpha, beta = 0.9, 0.6
    g = alpha * (q - beta * k * (k @ q))
    for i in range(dk):
        E = np.zeros((1, dk, dv))
        row = rng.standard_normal(dv)
        E[0, i] = row / np.linalg.norm(row)
        _, o = oracle.update_fp(E, q[None], k[None], np.zeros((1, dv)), [alpha], [beta])
        assert np.sum(o ** 2) == pytest.approx(g[i] ** 2, rel=1e-12, abs=1e-15)


# ---------------------------------------------------------------- quantizer (Eq. 3)
@pytest.mark.parametrize("b", [2, 4, 8])
def test_quantize_dequantize_idempotent(b):
    """Every code of every width survives dequantize -> quantize unchanged."""
    qb = 2 ** (b - 1) - 1
    rng = np.random.default_rng(b)
    dk, dv = 3, 2 * qb + 1
    codes = np.tile(np.arange(-qb, qb + 1, dtype=np.int8), (dk, 1))[None]
    r = rng.uniform(0.01, 2, (1, dk)).astype(np.float32)
    c = rng.uniform(0.01, 2, (1, dv)).astype(np.float32)
    bits = np.full((1, dk), b, np.uint8)
    S = oracle.dequant(codes, r, c, bits)
    assert np.array_equal(oracle.quantize(S, r, c, bits), codes)
    # the level set: S^ = r c q / q_b, so the extreme codes sit exactly at +-r c
    np.testing.assert_allclose(np.abs(S[0, :, 0]), r[0].astype(np.float64) * np.float64(c[0, 0]), rtol=1e-15)


def test_bruteforce_2x2_nearest_level():
    """On 2x2 tiles the oracle's codes minimise sum_i w_i^2 (X - X^)^2 over
    all joint code choices (enumerated for b <= 4) and are the per-entry
    nearest level for b = 8 (enumerating all 255 levels)."""
    rng = np.random.default_rng(5)
    for trial in range(40):
        bits = rng.choice([2, 4, 8], size=2).astype(np.uint8)
        r = rng.uniform(0.05, 1.0, 2).astype(np.float32)
        c = rng.uniform(0.05, 1.0, 2).astype(np.float32)
        X = rng.standard_normal((2, 2)) * 0.6
        w = rng.uniform(0.5, 2.0, 2)
        got = oracle.quantize(X[None], r[None], c[None], bits[None])[0]
        levels = [np.arange(-(2 ** (int(b) - 1) - 1), 2 ** (int(b) - 1)) for b in bits]
        if max(bits) <= 4:
            best, best_err = None, np.inf
            for z in itertools.product(levels[0], levels[0], levels[1], levels[1]):
                Z = np.array(z, dtype=np.float64).reshape(2, 2)
                qb = np.array([2 ** (int(b) - 1) - 1 for b in bits], np.float64)
                Xh = r[:, None].astype(np.float64) * c[None, :].astype(np.float64) * Z / qb[:, None]
                err = np.sum(w[:, None] ** 2 * (X - Xh) ** 2)
                if err < best_err:
                    best, best_err = Z, err
            assert np.array_equal(got, best.astype(np.int8))
        for i in range(2):
            qb = 2 ** (int(bits[i]) - 1) - 1
            for j in range(2):
                cand = float(r[i]) * float(c[j]) * levels[i] / qb
                assert got[i, j] == levels[i][np.argmin(np.abs(X[i, j] - cand))]


def test_quantizer_error_bound_and_clip():
    """|X^ - X| <= r c / (2 q_b) where X is in range; out of range clips to
    +-q_b (symmetric: -2^(b-1) is never produced)."""
    rng = np.random.default_rng(6)
    n, dk, dv = 4, 8, 8
    bits = rng.choice([2, 4, 8], size=(n, dk)).astype(np.uint8)
    r = rng.uniform(0.1, 1, (n, dk)).astype(np.float32)
    c = rng.uniform(0.1, 1, (n, dv)).astype(np.float32)
    X = rng.standard_normal((n, dk, dv)) * 1.5
    codes, y = oracle.quantize(X, r, c, bits, want_y=True)
    Xh = oracle.dequant(codes, r, c, bits)
    qb = (2.0 ** (bits.astype(np.int64) - 1) - 1)[:, :, None]
    rc = r.astype(np.float64)[:, :, None] * c.astype(np.float64)[:, None, :]
    inside = np.abs(y) <= qb
    assert np.all(np.abs(Xh - X)[inside] <= (rc / (2 * qb))[np.broadcast_to(inside, X.shape)] * (1 + 1e-12))
    assert np.all(codes[~inside] == np.sign(y[~inside]) * np.broadcast_to(qb, y.shape)[~inside])
    assert codes.min() >= -127


def test_ties_round_to_even():
    """Exact half-way values (power-of-two scales make X q_b/(r c) exact)
    round to the even neighbour."""
    b = 4                     # q_b = 7
    r = np.full((1, 1), 0.5, np.float32)
    c = np.full((1, 6), 2.0, np.float32)
    halfs = np.array([0.5, 1.5, 2.5, -0.5, -1.5, -6.5])
    X = (halfs / 7.0 * 1.0)[None, None, :]   # r c = 1
    codes, y = oracle.quantize(X, r, c, np.array([[b]], np.uint8), want_y=True)
    assert np.array_equal(y[0, 0], halfs)
    assert codes[0, 0].tolist() == [0, 2, 2, 0, -2, -6]


# ---------------------------------------------------------------- decode step (Table C2)
def test_decode_step_is_dequant_update_quantize():
    """The quantized step reads o from X before requantization (Eq. 4) and
    stores Q(X) (Eq. 3) on the frozen scales."""
    rng, S, q, k, v, alpha, beta = _case(7, n=3, dk=12, dv=10)
    bits = rng.choice([2, 4, 8], size=(3, 12)).astype(np.uint8)
    r, c = oracle.fit_absmax(S.astype(np.float32))
    codes = oracle.quantize(S, r, c, bits)
    new, o = oracle.decode_step(codes, r, c, bits, q, k, v, alpha, beta)
    X, o_ref = oracle.update_fp(oracle.dequant(codes, r, c, bits), q, k, v, alpha, beta)
    np.testing.assert_allclose(o, o_ref, rtol=0, atol=1e-14)
    assert np.array_equal(new, oracle.quantize(X, r, c, bits))
    # identity gate, no write: codes unchanged
    same, _ = oracle.decode_step(codes, r, c, bits, q, k, v, np.ones(3), np.zeros(3))
    assert np.array_equal(same, codes)


def test_error_propagation_proposition():
    """Proposition 1: with E_t = S^_t - S_t and eps_t = Q(X_t) - X_t,
    E_t = A_t E_{t-1} + eps_t and y^_t - y_t = E_{t-1}^T A_t^T q_t, and
    ||A_t||_2 <= 1 when |k| <= 1, 0 <= beta <= 1, 0 <= alpha <= 1."""
    rng = np.random.default_rng(8)
    n, dk, dv, T = 2, 16, 16, 6
    S = rng.standard_normal((n, dk, dv)) * 0.1
    bits = rng.choice([4, 8], size=(n, dk)).astype(np.uint8)
    r, c = oracle.fit_absmax(S.astype(np.float32))
    r = r * np.float32(3.0)                   # head-room so the trajectory rarely clips
    codes = oracle.quantize(S, r, c, bits)
    S_ref = S.copy()
    E_prev = oracle.dequant(codes, r, c, bits) - S_ref
    for t in range(T):
        q, k = _unit(rng, n, dk), _unit(rng, n, dk) * 0.9
        v = rng.standard_normal((n, dv)) * 0.1
        alpha, beta = rng.uniform(0.8, 1.0, n), rng.uniform(0, 1, n)
        Sh_prev = oracle.dequant(codes, r, c, bits)
        X, yhat = oracle.update_fp(Sh_prev, q, k, v, alpha, beta)
        codes, o_q = oracle.decode_step(codes, r, c, bits, q, k, v, alpha, beta)
        np.testing.assert_allclose(o_q, yhat, rtol=0, atol=1e-14)
        S_ref, y = oracle.update_fp(S_ref, q, k, v, alpha, beta)
        Sh = oracle.dequant(codes, r, c, bits)
        E = Sh - S_ref
        eps = Sh - X
        for b in range(n):
            A = (np.eye(dk) - beta[b] * np.outer(k[b], k[b])) * alpha[b]
            np.testing.assert_allclose(E[b], A @ E_prev[b] + eps[b], rtol=0, atol=1e-13)
            np.testing.assert_allclose(yhat[b] - y[b], E_prev[b].T @ A.T @ q[b], rtol=0, atol=1e-13)
            assert np.linalg.norm(A, 2) <= 1 + 1e-12
        E_prev = E


# ---------------------------------------------------------------- setup fit (Section 4.3)
def test_fit_absmax_bounds():
    """r_i = (m_i / w_i)^{1/2} with m_i the row mean |S|; r_i c_j >= |S_ij|
    everywhere, with equality (to fp32 rounding) at each column's arg-max."""
    rng = np.random.default_rng(9)
    S = (rng.standard_normal((3, 16, 12)) * np.exp(rng.standard_normal((3, 16, 1)))).astype(np.float32)
    w = rng.uniform(0.5, 2.0, (3, 16))
    r, c = oracle.fit_absmax(S, w)
    m = np.abs(S.astype(np.float64)).mean(axis=2)
    np.testing.assert_allclose(r.astype(np.float64) ** 2 * w, m, rtol=3e-7)
    rc = r.astype(np.float64)[:, :, None] * c.astype(np.float64)[:, None, :]
    assert np.all(rc >= np.abs(S))
    ratio = (np.abs(S) / rc).max(axis=1)
    np.testing.assert_allclose(ratio, 1.0, rtol=3e-7)
    # codes of the fitted state never clip, and each column reaches +-q_b
    bits = np.full((3, 16), 8, np.uint8)
    codes, y = oracle.quantize(S.astype(np.float64), r, c, bits, want_y=True)
    assert np.abs(y).max() <= 127.0
    assert np.all(np.abs(codes).max(axis=1) == 127)


def test_fit_zero_rows_use_floor():
    S = np.zeros((1, 4, 4), np.float32)
    S[0, 1, 2] = 0.25
    r, c = oracle.fit_absmax(S)
    assert r[0, 0] == np.float32(2.0 ** -60) and r[0, 1] > 0
    assert np.all(c > 0)


# ---------------------------------------------------------------- bit allocation (Eq. 6)
def test_mean_log_retention_closed_form():
    g = np.full((4, 3, 2), 0.9)
    g[..., 1] = 0.5
    np.testing.assert_allclose(oracle.mean_log_retention(g), [math.log(0.9), math.log(0.5)], rtol=1e-15)
    # half-life tau = log 2 / (-l) (Appendix B.4)
    assert math.log(2) / -math.log(0.5) == pytest.approx(1.0)


def test_lifetime_allocation_bruteforce():
    """The ranked allocation minimises sum_u L_u d(b_u) subject to the
    average-width budget (Eq. 6), checked by enumerating every assignment of
    {4, 8} to 2 rows x 4 heads with a shared distortion profile d(4) > d(8)."""
    rng = np.random.default_rng(10)
    for trial in range(5):
        H, dk, T, B = 4, 2, 6, 3
        gates = rng.uniform(0.6, 1.0, (T, B, H))
        bits = oracle.lifetime_bitmap(gates, dk, budget=6.0)
        ell = oracle.mean_log_retention(gates)
        Lw = np.array([oracle.lifetime_weight(e, 64) for e in ell])
        d = {4: 1.0, 8: 1.0 / 16}
        units = [(h, i) for h in range(H) for i in range(dk)]
        best = np.inf
        for choice in itertools.product([4, 8], repeat=len(units)):
            if sum(choice) > 6.0 * len(units):
                continue
            best = min(best, sum(Lw[h] * d[b] for (h, i), b in zip(units, choice)))
        got = sum(Lw[h] * d[int(bits[h, i])] for h, i in units)
        assert got == pytest.approx(best, rel=1e-12)
        assert bits.astype(float).mean() == 6.0


# ---------------------------------------------------------------- layout (include/stepq.h)
@pytest.mark.parametrize("b", [2, 4, 8])
def test_pack_single_field(b):
    """Each field lands in byte j of its row group at bit offset slot*b as a
    b-bit two's-complement integer, rows of one width in logical order."""
    dk, dv = 8, 128
    bits = np.full((1, dk), b, np.uint8)
    qb = 2 ** (b - 1) - 1
    rows_per_group = 8 // b
    for code in range(-qb, qb + 1):
        for i in (0, dk - 1, 3):
            j = (i * 37 + 5) % dv
            codes = np.zeros((1, 1, dk, dv), np.int8)
            codes[0, 0, i, j] = code
            r = np.zeros((1, 1, dk), np.float32)
            c = np.zeros((1, 1, dv), np.float32)
            img = oracle.pack_pool(codes, r, c, bits)
            g, s = i // rows_per_group, i % rows_per_group
            expect = ((code & ((1 << b) - 1)) << (s * b)) & 0xFF
            assert img[g * dv + j] == expect
            assert np.count_nonzero(img) == (1 if code != 0 else 0)


def test_pack_roundtrip_and_sizes():
    rng = np.random.default_rng(11)
    for dk, dv in [(64, 64), (128, 128), (32, 64)]:
        Hv, n = 3, 2
        bits = rng.choice([2, 4, 8], size=(Hv, dk)).astype(np.uint8)
        qb = (2 ** (bits.astype(np.int64) - 1) - 1)
        codes = rng.integers(-qb[None, :, :, None], qb[None, :, :, None] + 1, size=(n, Hv, dk, dv)).astype(np.int8)
        r = rng.uniform(0, 1, (n, Hv, dk)).astype(np.float32)
        c = rng.uniform(0, 1, (n, Hv, dv)).astype(np.float32)
        img = oracle.pack_pool(codes, r, c, bits)
        c2, r2, cc2 = oracle.unpack_pool(img, n, bits, dv)
        assert np.array_equal(c2, codes) and np.array_equal(r2, r) and np.array_equal(cc2, c)
        for h in range(Hv):
            n8, n4, n2 = [(bits[h] == w).sum() for w in (8, 4, 2)]
            groups = n8 + (n4 + 1) // 2 + (n2 + 3) // 4
            creg = -(-groups * dv // 128) * 128
            assert oracle.tile_bytes(bits[h], dv) == -(-(creg + 4 * dk + 4 * dv) // 128) * 128
        assert img.size == n * oracle.slot_bytes(bits, dv)


def test_six_bit_tile_bytes():
    """64 rows @8 + 64 rows @4 at d=128: 12,288 code bytes + 1,024 scale bytes."""
    bits = np.array([8] * 64 + [4] * 64, np.uint8)
    assert oracle.tile_bytes(bits, 128) == 13312
    bits = np.array([8] * 32 + [4] * 32 + [2] * 64, np.uint8)
    assert oracle.tile_bytes(bits, 128) == 8192 + 1024


# ---------------------------------------------------------------- the paper's printed accounting
def _gib(x):
    return x / 2 ** 30


def test_qwen_packed_bytes():
    g = GOLD
    assert oracle.packed_bytes_qwen6() == g["qwen6_packed_bytes"]["value"]
    assert oracle.packed_bytes_qwen6(pivot_scale_slots=True) == g["qwen6_compact_bytes_with_pivot_scale_slots"]["value"]
    fp32 = 4 * g["qwen_elements_per_request"]["value"]
    assert fp32 == g["qwen_state_bytes_fp32"]["value"]
    assert round(fp32 / oracle.packed_bytes_qwen6(), 2) == g["qwen6_ratio"]["value"]
    assert round(100 * (1 - oracle.packed_bytes_qwen6() / fp32), 2) == g["qwen6_reduction_pct"]["value"]
    assert round(oracle.compact_bits_qwen(6), 4) == g["b_qwen6"]["value"]


def test_kda_compact_sizes():
    g = GOLD
    N = g["kda_elements_per_request"]["value"]
    assert N == 20 * 32 * 128 * 128
    for bud, key_b, key_mib, key_ratio in [(6, "b_kda6", "kda6_mib", "kda6_ratio"), (4, "b_kda4", "kda4_mib", "kda4_ratio")]:
        b = oracle.compact_bits_kda(bud)
        assert round(b, 2) == g[key_b]["value"]
        mib = b * N / 8 / 2 ** 20
        assert mib == pytest.approx(g[key_mib]["value"], abs=1e-9)
        assert round(g["kda_fp32_mib"]["value"] / mib, 2) == g[key_ratio]["value"]


def test_serving_capacity_model():
    g = GOLD
    K = g["qwen_kv_bytes_per_token"]["value"]
    conv = g["qwen_conv_state_bytes"]["value"]
    S32 = g["qwen_state_bytes_fp32"]["value"] + conv
    Sq = g["qwen6_compact_bytes_with_pivot_scale_slots"]["value"] + conv
    assert Sq / 2 ** 20 == 31.4375
    # reserved state pool at B = 64 (weights and KV excluded)
    assert round(_gib(oracle.serving_memory(64, 0, 0, S32, K)), 2) == g["reserved_pool_fp32_b64_gib"]["value"]
    assert round(_gib(oracle.serving_memory(64, 0, 0, Sq, K)), 2) == g["reserved_pool_stepq_b64_gib"]["value"]
    # total serving memory at B = 512 with W4 weights, 128 + 1024 tokens
    W4 = g["qwen_weights_w4_bytes"]["value"]
    assert round(_gib(oracle.serving_memory(512, 1152, W4, S32, K)), 2) == g["qwen_total_w4_b512_fp32_gib"]["value"]
    assert round(_gib(oracle.serving_memory(512, 1152, W4, Sq, K)), 2) == g["qwen_total_w4_b512_stepq_gib"]["value"]
    # KDA recurrent-state pool at B = 512
    kda32 = g["kda_fp32_mib"]["value"] * 2 ** 20
    kda6 = g["kda6_mib"]["value"] * 2 ** 20
    assert round(_gib(oracle.serving_memory(512, 0, 0, kda32, 0)), 2) == g["kda_state_b512_fp32_gib"]["value"]
    assert round(_gib(oracle.serving_memory(512, 0, 0, kda6, 0)), 2) == g["kda_state_b512_stepq_gib"]["value"]
    # the FP32 pool first exceeds the BF16 weights at B = 70
    Wb = g["qwen_weights_bf16_bytes"]["value"]
    first = next(B for B in range(1, 1000) if (5 * B + 1) * S32 > Wb)
    assert first == g["fp32_pool_exceeds_bf16_weights_at_b"]["value"]


# ---------------------------------------------------------------- KDA channel-wise gate (Eq. 1, D = diag(d))
def _kda_case(seed=20, n=3, dk=12, dv=9):
    rng = np.random.default_rng(seed)
    S = rng.standard_normal((n, dk, dv)) * 0.3
    q, k = _unit(rng, n, dk), _unit(rng, n, dk)
    v = rng.standard_normal((n, dv))
    d = rng.uniform(0.3, 1.0, (n, dk))
    beta = rng.uniform(0.0, 1.0, n)
    return rng, S, q, k, v, d, beta


def test_kda_update_matches_affine_form():
    """Eq. 2 with D = diag(d): S_t = (I - beta k k^T) D S + beta k v^T."""
    _, S, q, k, v, d, beta = _kda_case()
    X, o = oracle.update_fp(S, q, k, v, d, beta)
    for t in range(S.shape[0]):
        A = (np.eye(S.shape[1]) - beta[t] * np.outer(k[t], k[t])) @ np.diag(d[t])
        Xr = A @ S[t] + beta[t] * np.outer(k[t], v[t])
        np.testing.assert_allclose(X[t], Xr, rtol=0, atol=1e-13)
        np.testing.assert_allclose(o[t], Xr.T @ q[t], rtol=0, atol=1e-13)
        assert np.linalg.norm(A, 2) <= np.max(d[t]) + 1e-12      # Proposition 1: ||A|| <= ||D|| <= 1


def test_kda_uniform_gate_is_gdn():
    """d_i = alpha for every row reproduces the scalar-gate path exactly."""
    _, S, q, k, v, d, beta = _kda_case(21)
    alpha = d[:, 0].copy()
    X1, o1 = oracle.update_fp(S, q, k, v, alpha, beta)
    X2, o2 = oracle.update_fp(S, q, k, v, np.repeat(alpha[:, None], S.shape[1], 1), beta)
    assert np.array_equal(X1, X2) and np.array_equal(o1, o2)


def test_kda_row_readout_sensitivity():
    """Eq. kda_sensitivity: g_i = d_i (q_i - beta k_i (k^T q)); a unit-norm
    error confined to key row i is read with squared norm g_i^2."""
    rng = np.random.default_rng(22)
    dk, dv = 10, 5
    q, k = _unit(rng, 1, dk)[0], _unit(rng, 1, dk)[0]
    d = rng.uniform(0.2, 1.0, dk)
    beta = 0.7
    g = d * (q - beta * k * (k @ q))
    for i in range(dk):
        E = np.zeros((1, dk, dv))
        row = rng.standard_normal(dv)
        E[0, i] = row / np.linalg.norm(row)
        _, o = oracle.update_fp(E, q[None], k[None], np.zeros((1, dv)), d[None], [beta])
        assert np.sum(o ** 2) == pytest.approx(g[i] ** 2, rel=1e-12, abs=1e-15)


def test_kda_decode_step_composition():
    rng, S, q, k, v, d, beta = _kda_case(23)
    bits = rng.choice([2, 4, 8], size=S.shape[:2]).astype(np.uint8)
    r, c = oracle.fit_absmax(S.astype(np.float32))
    codes = oracle.quantize(S, r, c, bits)
    new, o = oracle.decode_step(codes, r, c, bits, q, k, v, d, beta)
    X, o_ref = oracle.update_fp(oracle.dequant(codes, r, c, bits), q, k, v, d, beta)
    np.testing.assert_allclose(o, o_ref, rtol=0, atol=1e-14)
    assert np.array_equal(new, oracle.quantize(X, r, c, bits))
    same, _ = oracle.decode_step(codes, r, c, bits, q, k, v, np.ones_like(d), np.zeros_like(beta))
    assert np.array_equal(same, codes)


# ---------------------------------------------------------------- online dual-axis refit (Section 4.3, App. C)
def _refit_case(seed=30, n=4, dk=24, dv=10, kda=False):
    rng = np.random.default_rng(seed)
    bits = rng.choice([2, 4, 8], size=(n, dk)).astype(np.uint8)
    S = rng.standard_normal((n, dk, dv)) * np.exp(rng.standard_normal((n, dk, 1))) * 0.2
    r, c = oracle.fit_absmax(S.astype(np.float32))
    codes = oracle.quantize(S, r, c, bits)
    q, k = _unit(rng, n, dk), _unit(rng, n, dk)
    v = rng.standard_normal((n, dv))
    gate = rng.uniform(0.5, 1.0, (n, dk)) if kda else rng.uniform(0.5, 1.0, n)
    beta = rng.uniform(0.0, 1.0, n)
    w = np.exp(0.5 * rng.standard_normal((n, dk)))        # non-uniform row-impact factors
    return codes, r, c, bits, q, k, v, gate, beta, w


@pytest.mark.parametrize("kda", [False, True])
def test_refit_row_factors_closed_form(kda):
    """r'_i = (m_i / w_i)^{1/2} with m_i the mean |X_ij| of the updated state
    (Section 4.3), stored in fp32: r'^2 w = m up to that rounding."""
    codes, r, c, bits, q, k, v, g, beta, w = _refit_case(kda=kda)
    _, rn, _, _, ex = oracle.decode_step_refit(codes, r, c, bits, q, k, v, g, beta, w=w, want=("X",))
    m = np.abs(ex["X"]).mean(axis=2)
    np.testing.assert_allclose(rn.astype(np.float64) ** 2 * w, m, rtol=2.5e-7, atol=0)


@pytest.mark.parametrize("kda", [False, True])
def test_refit_column_fit_is_weighted_least_squares(kda):
    """With the fixed codes z (the rounded y0 / q_b), c'_j solves
    min_c sum_i w_i^2 (X_ij - r'_i c z_ij)^2: checked against a library
    least-squares solve of the weighted system, and against nearby c."""
    codes, r, c, bits, q, k, v, g, beta, w = _refit_case(seed=31, kda=kda)
    _, rn, cn, _, ex = oracle.decode_step_refit(codes, r, c, bits, q, k, v, g, beta, w=w, want=("X", "y0"))
    qb = (2.0 ** (bits.astype(np.int64) - 1) - 1)[:, :, None]
    z = np.clip(np.rint(ex["y0"]), -qb, qb) / qb
    X = ex["X"]
    n, dk, dv = X.shape
    for t in range(n):
        for j in range(dv):
            A = (w[t] * rn[t].astype(np.float64) * z[t, :, j])[:, None]
            bvec = w[t] * X[t, :, j]
            if not np.any(A):
                assert cn[t, j] == c[t, j]            # zero denominator: the previous scale stays
                continue
            sol = np.linalg.lstsq(A, bvec, rcond=None)[0][0]
            assert abs(float(cn[t, j]) - sol) <= 1e-7 * abs(sol)
            obj = lambda cc: float(np.sum((bvec - A[:, 0] * cc) ** 2))
            assert obj(sol) <= min(obj(sol * (1 + 1e-3)), obj(sol * (1 - 1e-3)))


def test_refit_fixed_codes_start_from_column_absmax():
    """The fixed codes come from the absmax column start: in every non-zero
    column the largest |y0_ij| / q_b is exactly 1, so no fixed code clips."""
    codes, r, c, bits, q, k, v, g, beta, w = _refit_case(seed=32)
    *_, ex = oracle.decode_step_refit(codes, r, c, bits, q, k, v, g, beta, w=w, want=("y0",))
    qb = (2.0 ** (bits.astype(np.int64) - 1) - 1)[:, :, None]
    ratio = np.abs(ex["y0"]) / qb
    np.testing.assert_allclose(ratio.max(axis=1), 1.0, rtol=0, atol=1e-12)


@pytest.mark.parametrize("kda", [False, True])
def test_refit_scale_invariance(kda):
    """Scaling the state and v by 4 scales X by 4: r' and c' double exactly
    (power-of-two scaling commutes with every rounding), the codes are
    unchanged and o scales by 4.  Scaling w by 4 halves r', doubles c' and
    keeps the codes."""
    codes, r, c, bits, q, k, v, g, beta, w = _refit_case(seed=33, kda=kda)
    base = oracle.decode_step_refit(codes, r, c, bits, q, k, v, g, beta, w=w)
    up = oracle.decode_step_refit(codes, 2 * r, 2 * c, bits, q, k, 4 * v, g, beta, w=w)
    assert np.array_equal(up[0], base[0])
    assert np.array_equal(up[1], 2 * base[1]) and np.array_equal(up[2], 2 * base[2])
    assert np.array_equal(up[3], 4 * base[3])
    ww = oracle.decode_step_refit(codes, r, c, bits, q, k, v, g, beta, w=4 * w)
    assert np.array_equal(ww[0], base[0])
    assert np.array_equal(ww[1], base[1] / 2) and np.array_equal(ww[2], 2 * base[2])


def test_refit_zero_row_and_zero_column():
    """A row with k_i = 0 and zero codes stays zero: r' falls to the 2^-60
    floor.  A column with zero codes and v_j = 0 stays zero: its denominator
    is zero and the previous scale is kept (Appendix C.1)."""
    codes, r, c, bits, q, k, v, g, beta, w = _refit_case(seed=34)
    codes[:, 3, :] = 0
    k[:, 3] = 0.0
    codes[:, :, 5] = 0
    v[:, 5] = 0.0
    out, rn, cn, _ = oracle.decode_step_refit(codes, r, c, bits, q, k, v, g, beta, w=w)
    assert np.all(rn[:, 3] == np.float32(2.0 ** -60)) and np.all(out[:, 3, :] == 0)
    assert np.array_equal(cn[:, 5], c[:, 5]) and np.all(out[:, :, 5] == 0)


def test_refit_requantizes_with_the_new_scales():
    """Final codes are the quantizer (Eq. 3, pinned above) applied to X with
    the refitted scales; the readout is taken before, so it equals the
    frozen-scale step's readout (Table C2, step 3 precedes steps 4-6)."""
    codes, r, c, bits, q, k, v, g, beta, w = _refit_case(seed=35)
    out, rn, cn, o, ex = oracle.decode_step_refit(codes, r, c, bits, q, k, v, g, beta, w=w, want=("X",))
    assert np.array_equal(out, oracle.quantize(ex["X"], rn, cn, bits))
    _, o_frozen = oracle.decode_step(codes, r, c, bits, q, k, v, g, beta)
    assert np.array_equal(o, o_frozen)


@pytest.mark.parametrize("levels", [oracle.LEVELS_ABSMAX, oracle.LEVELS_POW2])
def test_refit_column_range_encloses_every_tie_rounding(levels):
    """The (lo, hi) column-factor range encloses the least-squares factor of
    every combination of other roundings of the near-tie fixed codes,
    enumerated here and solved with a library least-squares routine; with a
    zero window the range is the factor itself.  Both level normalisations
    (a code q of a b-bit row is the level q / q_b, or 2^(8-b) q)."""
    codes, r, c, bits, q, k, v, g, beta, w = _refit_case(seed=36, n=2, dk=10, dv=6)
    win = 0.15                                   # wide, so that several codes per column qualify
    _, rn, cn, _, ex = oracle.decode_step_refit(codes, r, c, bits, q, k, v, g, beta, w=w,
                                                want=("X", "y0", "c_range"), tie_window=win, levels=levels)
    lo, hi = ex["c_range"]
    qb = (2.0 ** (bits.astype(np.int64) - 1) - 1)[:, :, None]
    lev = 1.0 / qb if levels == oracle.LEVELS_ABSMAX else (2.0 ** (8 - bits.astype(np.int64)))[:, :, None]
    y0, X = ex["y0"], ex["X"]
    z = np.clip(np.rint(y0), -qb, qb)
    n_multi = 0
    for t in range(X.shape[0]):
        for j in range(X.shape[2]):
            a = np.abs(y0[t, :, j])
            near = [i for i in range(X.shape[1]) if abs(a[i] - np.floor(a[i]) - 0.5) <= win]
            alts = []
            for i in near:
                alt = z[t, i, j] - 1 if z[t, i, j] > y0[t, i, j] else z[t, i, j] + 1
                if abs(alt) <= qb[t, i, 0]:
                    alts.append((i, alt))
            n_multi += len(alts) > 1
            for mask in itertools.product([0, 1], repeat=len(alts)):
                zz = z[t, :, j].copy()
                for (i, alt), m in zip(alts, mask):
                    if m:
                        zz[i] = alt
                A = (w[t] * rn[t].astype(np.float64) * zz * lev[t, :, 0])[:, None]
                if not np.any(A):
                    continue
                cs = np.linalg.lstsq(A, w[t] * X[t, :, j], rcond=None)[0][0]
                assert lo[t, j] * (1 - 1e-12) <= cs <= hi[t, j] * (1 + 1e-12)
            assert lo[t, j] <= cn[t, j] * (1 + 1e-7) and cn[t, j] <= hi[t, j] * (1 + 1e-7)
    assert n_multi > 0
    *_, ex0 = oracle.decode_step_refit(codes, r, c, bits, q, k, v, g, beta, w=w, want=("c_range",), tie_window=0.0,
                                       levels=levels)
    lo0, hi0 = ex0["c_range"]
    assert np.array_equal(lo0, hi0) and np.array_equal(lo0.astype(np.float32), cn)


# ---------------------------------------------------------------- row-wise absmax INT-b baseline (Section 5.1)
@pytest.mark.parametrize("kda", [False, True])
def test_rowmax_baseline_closed_form(kda):
    """r'_i is the row's largest |X_ij| (computed here from X of the pinned
    update), c' = 1, the largest entry of every row lands on +-q_b, and no
    entry is off by more than half a level r'/(2 q_b)."""
    codes, r, c, bits, q, k, v, g, beta, _ = _refit_case(seed=40, kda=kda)
    out, rn, cn, o = oracle.decode_step_rowmax(codes, r, c, bits, q, k, v, g, beta)
    S = oracle.dequant(codes, r, c, bits)
    X, o_ref = oracle.update_fp(S, q, k, v, g, beta)
    np.testing.assert_allclose(rn, np.abs(X).max(axis=2), rtol=6e-8, atol=0)
    assert np.all(cn == 1.0)
    qb = (2.0 ** (bits.astype(np.int64) - 1) - 1)[:, :, None]
    am = np.abs(X).argmax(axis=2)
    top = np.take_along_axis(out, am[:, :, None], axis=2)[:, :, 0]
    assert np.array_equal(np.abs(top), qb[:, :, 0].astype(np.int8))
    Xh = rn.astype(np.float64)[:, :, None] * out / qb
    assert np.all(np.abs(Xh - X) <= rn.astype(np.float64)[:, :, None] / (2 * qb) * (1 + 1e-6))
    assert np.array_equal(o, o_ref)


def test_rowmax_baseline_is_refit_free_of_columns():
    """With all column factors 1 the row-absmax requantization is the
    quantizer (pinned above) with r = row max and c = 1; scaling a row of
    the state scales its r' and leaves its codes (power of two: exactly)."""
    codes, r, c, bits, q, k, v, g, beta, _ = _refit_case(seed=41)
    out, rn, cn, _, y = oracle.decode_step_rowmax(codes, r, c, bits, q, k, v, g, beta, want_y=True)
    S = oracle.dequant(codes, r, c, bits)
    X, _ = oracle.update_fp(S, q, k, v, g, beta)
    assert np.array_equal(out, oracle.quantize(X, rn, cn, bits))
    up = oracle.decode_step_rowmax(codes, 4 * r, c, bits, q, k, 4 * v, g, beta)
    assert np.array_equal(up[0], out) and np.array_equal(up[1], 4 * rn)


# ---------------------------------------------------------------- FP16 pivot rows (Section 3.2, Table C1)
def test_binary16_conversions_match_ieee():
    """The oracle's binary16 decoding of every bit pattern, and its rounding
    of doubles (ties to even, subnormals, overflow), agree with numpy's
    IEEE half type."""
    h = np.arange(65536, dtype=np.uint16)
    ref = h.view(np.float16).astype(np.float64)
    got = oracle.half_to_double(h)
    fin = ~np.isnan(ref)
    assert np.array_equal(got[fin], ref[fin]) and np.all(np.isnan(got[~fin]))
    rng = np.random.default_rng(50)
    vals = np.unique(ref[np.isfinite(ref)])
    x = np.concatenate([
        rng.standard_normal(20000) * np.exp(rng.uniform(-20, 12, 20000)),
        vals[:-1] + 0.5 * np.diff(vals),                  # exact midpoints between neighbours
        np.array([65504.0, 65519.99, 65520.0, 1e6, -65520.0, 2.0 ** -25, 2.0 ** -24, 3 * 2.0 ** -26, 0.0, -0.0]),
    ])
    x = x[np.isfinite(x)]
    with np.errstate(over="ignore"):
        want = x.astype(np.float16).view(np.uint16)
    assert np.array_equal(oracle.double_to_half(x), want)


def _pivot_map(rng, n, dk, n_piv):
    bits = rng.choice([2, 4, 8], size=(n, dk)).astype(np.uint8)
    for t in range(n):
        bits[t, rng.choice(dk, size=n_piv, replace=False)] = 16
    return bits


def test_pivot_layout_placement_and_roundtrip():
    """A pivot row's binary16 values sit after the codes region, in physical
    order, little-endian; the integer rows and scales are unaffected; pack
    and unpack are inverse."""
    dk, dv = 10, 64
    bits = np.array([[8, 16, 4, 2, 16, 8, 4, 4, 2, 2]], np.uint8)
    codes = np.zeros((1, 1, dk, dv), np.int8)
    pv = np.zeros((1, 1, dk, dv), np.uint16)
    pv[0, 0, 4, 3] = 0xBEEF                           # second pivot row, column 3
    r = np.arange(1, dk + 1, dtype=np.float32)[None, None]
    c = np.full((1, 1, dv), 0.5, np.float32)
    img = oracle.pack_pool(codes, r, c, bits, pv=pv)
    groups = 2 + 2 + 1                                # two 8-bit rows, three 4-bit rows, three 2-bit rows
    creg = ((groups * dv + 127) // 128) * 128
    piv = img[creg:creg + 2 * 2 * dv]
    nz = np.nonzero(piv)[0]
    assert list(nz) == [2 * dv + 6, 2 * dv + 7] and piv[2 * dv + 6] == 0xEF and piv[2 * dv + 7] == 0xBE
    rr = img[creg + 4 * dv: creg + 4 * dv + 4 * dk].view(np.float32)
    assert list(rr) == [2, 5, 1, 6, 3, 7, 8, 4, 9, 10]   # physical order: pivots, 8, 4, 2
    assert len(img) == oracle.slot_bytes(bits, dv) == ((creg + 4 * dv + 4 * (dk + dv) + 127) // 128) * 128
    rng = np.random.default_rng(51)
    bits2 = _pivot_map(rng, 3, 20, 3)
    qb = 2 ** (bits2.astype(np.int64) - 1) - 1
    codes2 = np.where(bits2[None, :, :, None] == 16, 0,
                      rng.integers(-qb[None, :, :, None], qb[None, :, :, None] + 1, size=(2, 3, 20, 64))).astype(np.int8)
    pv2 = rng.integers(0, 65536, size=(2, 3, 20, 64)).astype(np.uint16) * (bits2[None, :, :, None] == 16)
    r2 = rng.uniform(0.1, 1, (2, 3, 20)).astype(np.float32)
    c2 = rng.uniform(0.1, 1, (2, 3, 64)).astype(np.float32)
    back = oracle.unpack_pool(oracle.pack_pool(codes2, r2, c2, bits2, pv=pv2), 2, bits2, 64)
    assert np.array_equal(back[0], codes2) and np.array_equal(back[3], pv2)
    assert np.array_equal(back[1], r2) and np.array_equal(back[2], c2)


@pytest.mark.parametrize("kda", [False, True])
def test_pivot_decode_is_update_then_binary16(kda):
    """Pivot rows enter the update with their binary16 values and leave as X
    rounded to binary16 (pinned conversion); integer rows follow the pinned
    quantizer; o is read from X as without pivots."""
    rng = np.random.default_rng(52)
    n, dk, dv = 3, 16, 12
    bits = _pivot_map(rng, n, dk, 2)
    S = rng.standard_normal((n, dk, dv)) * 0.3
    r, c = oracle.fit_absmax(S.astype(np.float32), bits=bits)
    codes, pv = oracle.quantize(S, r, c, bits)
    np.testing.assert_array_equal(oracle.half_to_double(pv)[bits == 16], oracle.half_to_double(
        oracle.double_to_half(S))[bits == 16])
    q, k = _unit(rng, n, dk), _unit(rng, n, dk)
    v = rng.standard_normal((n, dv))
    g = rng.uniform(0.5, 1, (n, dk)) if kda else rng.uniform(0.5, 1, n)
    beta = rng.uniform(0, 1, n)
    out, o, pv2 = oracle.decode_step(codes, r, c, bits, q, k, v, g, beta, pv=pv)
    Sh = oracle.dequant(codes, r, c, bits, pv=pv)
    X, o_ref = oracle.update_fp(Sh, q, k, v, g, beta)
    assert np.array_equal(o, o_ref)
    assert np.array_equal(pv2[bits == 16], oracle.double_to_half(X)[bits == 16])
    want, _ = oracle.quantize(X, r, c, bits)
    assert np.array_equal(out, want) and np.all(out[bits == 16] == 0)


@pytest.mark.parametrize("mode", ["refit", "rowmax"])
def test_pivots_take_no_part_in_the_scale_fits(mode):
    """With k = 0 on the pivot rows they do not feed the other rows' update,
    so the refit of the integer rows must equal the refit of the tile with
    the pivot rows removed, bit for bit, however large the pivot values
    (Appendix C.1 fits the non-pivot integer rows)."""
    rng = np.random.default_rng(53 if mode == "refit" else 54)
    n, dk, dv = 2, 14, 10
    bits = np.tile(np.array([[8, 16, 4, 8, 2, 16, 4, 8, 8, 4, 2, 16, 8, 4]], np.uint8), (n, 1))
    keep = bits[0] != 16
    S = rng.standard_normal((n, dk, dv)) * 0.2
    S[:, ~keep, :] *= 1e3                                      # outlier pivot rows
    r, c = oracle.fit_absmax(S.astype(np.float32), bits=bits)
    r_int, c_int = oracle.fit_absmax(S[:, keep].astype(np.float32))
    assert np.array_equal(c, c_int) and np.array_equal(r[:, keep], r_int)
    codes, pv = oracle.quantize(S, r, c, bits)
    q, k = _unit(rng, n, dk), _unit(rng, n, dk)
    k[:, ~keep] = 0.0
    v = rng.standard_normal((n, dv))
    g = rng.uniform(0.5, 1, n)
    beta = rng.uniform(0, 1, n)
    w = np.exp(0.3 * rng.standard_normal((n, dk)))
    if mode == "refit":
        full = oracle.decode_step_refit(codes, r, c, bits, q, k, v, g, beta, w=w, pv=pv)
        part = oracle.decode_step_refit(codes[:, keep], r[:, keep], c, bits[:, keep], q[:, keep], k[:, keep], v, g,
                                        beta, w=w[:, keep])
    else:
        full = oracle.decode_step_rowmax(codes, r, c, bits, q, k, v, g, beta, pv=pv)
        part = oracle.decode_step_rowmax(codes[:, keep], r[:, keep], c, bits[:, keep], q[:, keep], k[:, keep], v,
                                         g, beta)
    assert np.array_equal(full[0][:, keep], part[0])
    assert np.array_equal(full[1][:, keep], part[1]) and np.array_equal(full[2], part[2])
    assert np.array_equal(full[1][:, ~keep], r[:, ~keep])       # pivots keep their (unused) row factor
