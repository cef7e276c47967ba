"""fp64 reference oracle for the quantized gated-Delta decode step.

TEST INFRASTRUCTURE ONLY: imported by tests/, by ``__graft_entry__.smoke()``
and by the ``cpu_baseline`` leg of ``bench.py``, never by the product package.
It shares no code with the HIP path (the two meet only through the seeded
workload draws, which hold none of the method's arithmetic).

The numeric work is in ``stepq_oracle.c`` (plain loops, double precision);
this module marshals numpy arrays to it and holds the setup-side steps that
are small enough to be plain Python: the lifetime-ranked bit allocation and
the paper's storage accounting.

Parity status of each function (what pins it) is listed in the tests that
exercise it; the whole-trajectory output is "parity unpinned" against the
paper, which prints no state values.
"""
from __future__ import annotations

import ctypes
import math
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "stepq_oracle.c")
_LIB_PATH = os.path.join(_HERE, "libstepq_oracle.so")
_lib = None


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (-O2, OpenMP, no FP contraction)."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-ffp-contract=off", "-fno-fast-math",
                               "-shared", "-fPIC", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build()
        L = ctypes.CDLL(_LIB_PATH)
        P = ctypes.c_void_p
        i = ctypes.c_int
        L.orc_fit_absmax.argtypes = [i, i, i, P, P, P, P, P, i]
        L.orc_quantize.argtypes = [i, i, i, P, P, P, P, P, P, P, i]
        L.orc_dequant.argtypes = [i, i, i, P, P, P, P, P, P, i]
        L.orc_update_fp.argtypes = [i, i, i, P, P, P, P, P, i, P, P, P]
        L.orc_decode_step.argtypes = [i, i, i, P, P, P, P, P, P, P, P, i, P, P, P, P, P, P, i]
        L.orc_decode_step_refit.argtypes = [i, i, i, P, P, P, P, P, P, P, P, P, i, P, P, P, P, P, P, P, P,
                                            ctypes.c_double, P, P, P, P, i]
        L.orc_decode_step_rowmax.argtypes = [i, i, i, P, P, P, P, P, P, P, P, i, P, P, P, P, P, P, P, P, i]
        L.orc_fit_dual_axis.argtypes = [i, i, i, P, P, P, P, P, P, P]
        L.orc_half_to_double.argtypes = [ctypes.c_size_t, P, P]
        L.orc_double_to_half.argtypes = [ctypes.c_size_t, P, P]
        L.orc_tile_bytes.argtypes = [i, i, P]
        L.orc_tile_bytes.restype = ctypes.c_size_t
        L.orc_slot_bytes.argtypes = [i, i, i, P]
        L.orc_slot_bytes.restype = ctypes.c_size_t
        L.orc_pack_pool.argtypes = [i, i, i, i, P, P, P, P, P, P]
        L.orc_unpack_pool.argtypes = [i, i, i, i, P, P, P, P, P, P]
        L.orc_max_threads.restype = ctypes.c_int
        L.orc_set_threads.argtypes = [ctypes.c_int]
        L.orc_set_threads.restype = None
        _lib = L
    return _lib


def _p(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p) if a is not None else None


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


def max_threads() -> int:
    return int(lib().orc_max_threads())


def set_threads(n: int) -> None:
    """Threads of the oracle's tile loops from now on (timing only)."""
    lib().orc_set_threads(int(n))


# Level normalisation of the stored integers (Section 4.3, Appendix C.1):
# levels 0 (N1) z = q / q_b; levels 1 (N2) z = 2^(8-b) q, the paper's KDA
# codebook.  Every numeric entry point below takes it (default N1).
LEVELS_ABSMAX, LEVELS_POW2 = 0, 1


def _lv(levels) -> int:
    if levels not in (LEVELS_ABSMAX, LEVELS_POW2):
        raise ValueError("levels must be 0 (N1: q / q_b) or 1 (N2: 2^(8-b) q)")
    return int(levels)


# FP16 pivot rows (width 16): their values travel as binary16 bit patterns,
# pv [n][dk][dv] uint16 (only pivot rows read or written).  Every function
# below that takes a bit map with pivot rows needs pv and returns the new pv
# as its last result.
def _has_pivots(bits) -> bool:
    return bool(np.any(np.asarray(bits) == 16))


def _pv_in(pv, bits, shape):
    if not _has_pivots(bits):
        return None
    if pv is None:
        raise ValueError("the bit map has pivot rows: pass their binary16 values as pv")
    return _c(np.broadcast_to(pv, shape), np.uint16)


def half_to_double(h):
    h = _c(h, np.uint16)
    out = np.empty(h.shape, np.float64)
    lib().orc_half_to_double(h.size, _p(h), _p(out))
    return out


def double_to_half(x):
    x = _c(x, np.float64)
    out = np.empty(x.shape, np.uint16)
    lib().orc_double_to_half(x.size, _p(x), _p(out))
    return out


# ---------------------------------------------------------------------------
# numeric entry points (shapes: tiles flattened to a leading n)
def fit_absmax(S, w=None, bits=None, levels=LEVELS_ABSMAX):
    """Setup fit (Section 4.3 row factors, absmax column factor).
    S: [n][dk][dv] float32 -> (r [n][dk], c [n][dv]) float32.  bits
    (optional under N1, needed under N2, whose largest level depends on
    the width): pivot rows (16) are left out of the column factor."""
    if _lv(levels) and bits is None:
        raise ValueError("the N2 fit needs the row widths")
    S = _c(S, np.float32)
    n, dk, dv = S.shape
    r = np.empty((n, dk), np.float32)
    c = np.empty((n, dv), np.float32)
    wv = None if w is None else _c(np.broadcast_to(w, (n, dk)), np.float64)
    bt = None if bits is None else _c(np.broadcast_to(bits, (n, dk)), np.uint8)
    lib().orc_fit_absmax(n, dk, dv, _p(S), _p(wv), _p(bt), _p(r), _p(c), _lv(levels))
    return r, c


def quantize(X, r, c, bits, want_y=False, levels=LEVELS_ABSMAX):
    """Eq. 3 on the dual-axis representation. X [n][dk][dv] (fp64),
    bits [n][dk] -> int8 codes (and the unrounded values if want_y)."""
    X = _c(X, np.float64)
    n, dk, dv = X.shape
    r, c, bits = _c(r, np.float32), _c(c, np.float32), _c(np.broadcast_to(bits, (n, dk)), np.uint8)
    codes = np.empty((n, dk, dv), np.int8)
    y = np.empty((n, dk, dv), np.float64) if want_y else None
    pv = np.zeros((n, dk, dv), np.uint16) if _has_pivots(bits) else None
    lib().orc_quantize(n, dk, dv, _p(X), _p(r), _p(c), _p(bits), _p(codes), _p(y), _p(pv), _lv(levels))
    out = (codes, y) if want_y else (codes,)
    out = out + ((pv,) if pv is not None else ())
    return out if len(out) > 1 else out[0]


def dequant(codes, r, c, bits, pv=None, levels=LEVELS_ABSMAX):
    codes = _c(codes, np.int8)
    n, dk, dv = codes.shape
    r, c, bits = _c(r, np.float32), _c(c, np.float32), _c(np.broadcast_to(bits, (n, dk)), np.uint8)
    pvi = _pv_in(pv, bits, (n, dk, dv))
    S = np.empty((n, dk, dv), np.float64)
    lib().orc_dequant(n, dk, dv, _p(codes), _p(r), _p(c), _p(bits), _p(pvi), _p(S), _lv(levels))
    return S


def _gates(alpha, n, dk):
    """alpha [n] (scalar gate, GDN) or [n][dk] (channel-wise gate, KDA)."""
    a = _c(alpha, np.float64)
    if a.size == n:
        return a.reshape(n), 0
    return a.reshape(n, dk), 1


def update_fp(S, q, k, v, alpha, beta):
    """Eq. 1 with D = alpha I (alpha [n]) or D = diag(d) (alpha [n][dk]) on a
    real state; readout from X (Eq. 4)."""
    S = _c(S, np.float64)
    n, dk, dv = S.shape
    q, k, v = _c(q, np.float64), _c(k, np.float64), _c(v, np.float64)
    a, per_row = _gates(alpha, n, dk)
    beta = _c(beta, np.float64).reshape(n)
    X = np.empty_like(S)
    o = np.empty((n, dv), np.float64)
    lib().orc_update_fp(n, dk, dv, _p(S), _p(q), _p(k), _p(v), _p(a), per_row, _p(beta), _p(X), _p(o))
    return X, o


def decode_step(codes, r, c, bits, q, k, v, alpha, beta, want_y=False, pv=None, levels=LEVELS_ABSMAX):
    """One quantized decode step with frozen scales (Table C2 steps 1-3, 6);
    alpha [n] for the GDN gate or [n][dk] for the KDA channel-wise gate."""
    codes = _c(codes, np.int8)
    n, dk, dv = codes.shape
    r, c, bits = _c(r, np.float32), _c(c, np.float32), _c(np.broadcast_to(bits, (n, dk)), np.uint8)
    q, k, v = _c(q, np.float64), _c(k, np.float64), _c(v, np.float64)
    a, per_row = _gates(alpha, n, dk)
    beta = _c(beta, np.float64).reshape(n)
    out = np.empty_like(codes)
    o = np.empty((n, dv), np.float64)
    y = np.empty((n, dk, dv), np.float64) if want_y else None
    pvi = _pv_in(pv, bits, (n, dk, dv))
    pvo = np.zeros((n, dk, dv), np.uint16) if pvi is not None else None
    lib().orc_decode_step(n, dk, dv, _p(codes), _p(r), _p(c), _p(bits), _p(q), _p(k), _p(v),
                          _p(a), per_row, _p(beta), _p(out), _p(o), _p(y), _p(pvi), _p(pvo), _lv(levels))
    res = (out, o, y) if want_y else (out, o)
    return res + (pvo,) if pvo is not None else res


def decode_step_refit(codes, r, c, bits, q, k, v, alpha, beta, w=None, want=(), tie_window=2e-3, pv=None,
                      levels=LEVELS_ABSMAX):
    """One quantized decode step with the online dual-axis refit (Table C2
    steps 1-6, Section 4.3, Appendix C.1).  Returns (codes, r, c, o) with the
    new fp32 scales, plus a dict of the requested extras among "y", "y0", "X"
    and "c_range" (the (lo, hi) column-factor bounds over the other roundings
    of fixed codes within tie_window of a rounding boundary).
    w: row-impact factors [n][dk] (None: 1)."""
    codes = _c(codes, np.int8)
    n, dk, dv = codes.shape
    r, c, bits = _c(r, np.float32), _c(c, np.float32), _c(np.broadcast_to(bits, (n, dk)), np.uint8)
    q, k, v = _c(q, np.float64), _c(k, np.float64), _c(v, np.float64)
    a, per_row = _gates(alpha, n, dk)
    beta = _c(beta, np.float64).reshape(n)
    wt = None if w is None else _c(np.broadcast_to(w, (n, dk)), np.float64)
    out = np.empty_like(codes)
    r_out = np.empty((n, dk), np.float32)
    c_out = np.empty((n, dv), np.float32)
    o = np.empty((n, dv), np.float64)
    extra = {key: np.empty((n, dk, dv), np.float64) for key in want if key != "c_range"}
    lo = hi = None
    if "c_range" in want:
        lo, hi = np.empty((n, dv), np.float64), np.empty((n, dv), np.float64)
        if "y0" not in extra:
            extra["y0"] = np.empty((n, dk, dv), np.float64)
    pvi = _pv_in(pv, bits, (n, dk, dv))
    pvo = np.zeros((n, dk, dv), np.uint16) if pvi is not None else None
    lib().orc_decode_step_refit(n, dk, dv, _p(codes), _p(r), _p(c), _p(bits), _p(wt), _p(q), _p(k), _p(v),
                                _p(a), per_row, _p(beta), _p(out), _p(r_out), _p(c_out), _p(o),
                                _p(extra.get("y")), _p(extra.get("y0")), _p(extra.get("X")), float(tie_window),
                                _p(lo), _p(hi), _p(pvi), _p(pvo), _lv(levels))
    if lo is not None:
        extra["c_range"] = (lo, hi)
    res = (out, r_out, c_out, o, extra) if want else (out, r_out, c_out, o)
    return res + (pvo,) if pvo is not None else res


def decode_step_rowmax(codes, r, c, bits, q, k, v, alpha, beta, want_y=False, pv=None, levels=LEVELS_ABSMAX):
    """One decode step of the row-wise absmax INT-b baseline (Section 5.1) on
    the same quantized tile: returns (codes, r, c, o[, y]) with r'_i =
    max_j |X_ij| and c' = 1."""
    codes = _c(codes, np.int8)
    n, dk, dv = codes.shape
    r, c, bits = _c(r, np.float32), _c(c, np.float32), _c(np.broadcast_to(bits, (n, dk)), np.uint8)
    q, k, v = _c(q, np.float64), _c(k, np.float64), _c(v, np.float64)
    a, per_row = _gates(alpha, n, dk)
    beta = _c(beta, np.float64).reshape(n)
    out = np.empty_like(codes)
    r_out = np.empty((n, dk), np.float32)
    c_out = np.empty((n, dv), np.float32)
    o = np.empty((n, dv), np.float64)
    y = np.empty((n, dk, dv), np.float64) if want_y else None
    pvi = _pv_in(pv, bits, (n, dk, dv))
    pvo = np.zeros((n, dk, dv), np.uint16) if pvi is not None else None
    lib().orc_decode_step_rowmax(n, dk, dv, _p(codes), _p(r), _p(c), _p(bits), _p(q), _p(k), _p(v), _p(a),
                                 per_row, _p(beta), _p(out), _p(r_out), _p(c_out), _p(o), _p(y), _p(pvi), _p(pvo),
                                 _lv(levels))
    res = (out, r_out, c_out, o, y) if want_y else (out, r_out, c_out, o)
    return res + (pvo,) if pvo is not None else res


def tile_bytes(bits_row, d_v: int) -> int:
    b = _c(bits_row, np.uint8)
    return int(lib().orc_tile_bytes(b.shape[0], d_v, _p(b)))


def slot_bytes(bits, d_v: int) -> int:
    bits = _c(bits, np.uint8)
    Hv, dk = bits.shape
    return int(lib().orc_slot_bytes(Hv, dk, d_v, _p(bits)))


def pack_pool(codes, r, c, bits, pv=None):
    """Pool image (bytes) per the layout definition. codes [S][Hv][dk][dv];
    pv [S][Hv][dk][dv] binary16 values of pivot rows (if the map has any)."""
    codes = _c(codes, np.int8)
    S, Hv, dk, dv = codes.shape
    r, c, bits = _c(r, np.float32), _c(c, np.float32), _c(bits, np.uint8)
    pvi = _pv_in(pv, bits, codes.shape)
    out = np.zeros(S * slot_bytes(bits, dv), np.uint8)
    lib().orc_pack_pool(S, Hv, dk, dv, _p(bits), _p(codes), _p(pvi), _p(r), _p(c), _p(out))
    return out


def unpack_pool(pool, n_slots, bits, d_v):
    """(codes, r, c[, pv]) of a pool image; pv only if the map has pivots."""
    bits = _c(bits, np.uint8)
    Hv, dk = bits.shape
    pool = _c(pool, np.uint8)
    codes = np.empty((n_slots, Hv, dk, d_v), np.int8)
    r = np.empty((n_slots, Hv, dk), np.float32)
    c = np.empty((n_slots, Hv, d_v), np.float32)
    pv = np.zeros((n_slots, Hv, dk, d_v), np.uint16) if _has_pivots(bits) else None
    lib().orc_unpack_pool(n_slots, Hv, dk, d_v, _p(bits), _p(pool), _p(codes), _p(pv), _p(r), _p(c))
    return (codes, r, c, pv) if pv is not None else (codes, r, c)


def fit_dual_axis(X, bits, w=None):
    """Key-Row-Aware Dual-Axis fit of states X [n][dk][dv] (fp64): returns
    (codes, r, c[, pv]) -- the spatial codec of Section 4.3 / Appendix C.1."""
    X = _c(X, np.float64)
    n, dk, dv = X.shape
    bits = _c(np.broadcast_to(bits, (n, dk)), np.uint8)
    wt = None if w is None else _c(np.broadcast_to(w, (n, dk)), np.float64)
    r = np.empty((n, dk), np.float32)
    c = np.empty((n, dv), np.float32)
    codes = np.empty((n, dk, dv), np.int8)
    pv = np.zeros((n, dk, dv), np.uint16) if _has_pivots(bits) else None
    lib().orc_fit_dual_axis(n, dk, dv, _p(X), _p(bits), _p(wt), _p(r), _p(c), _p(codes), _p(pv))
    return (codes, r, c, pv) if pv is not None else (codes, r, c)


# ---------------------------------------------------------------------------
# setup side: lifetime-aware bit allocation (Section 3.2, Eq. 6)
def mean_log_retention(gates) -> np.ndarray:
    """l_u = E_cal[log r_{t,u}] (Appendix A.3, Eq. calibration_lifetime).
    gates: [T][B][H] -> l per head [H], averaging over steps and requests."""
    g = np.asarray(gates, np.float64)
    T, B, H = g.shape
    out = np.zeros(H)
    for h in range(H):
        s = 0.0
        for t in range(T):
            for b in range(B):
                s += math.log(g[t, b, h])
        out[h] = s / (T * B)
    return out


def lifetime_weight(ell: float, horizon: int) -> float:
    """L_u = sum_{j=0}^{H-1} exp(2 j l_u) (Section 3.2)."""
    return sum(math.exp(2.0 * j * ell) for j in range(horizon))


def lifetime_bitmap(gates, d_k: int, budget: float = 6.0, lo: int = 4, hi: int = 8) -> np.ndarray:
    """Key-row widths from two candidates under an average budget.

    Units are key rows (n_u = d_v elements each, equal for all units).  With
    one distortion profile d(b) shared by all units, the objective of Eq. 6,
    sum_u L_u d(b_u), is minimised by giving the wider code to the units of
    largest L_u, i.e. of largest mean log retention l_u (L_u is increasing in
    l_u).  The budget admits floor(N (budget - lo) / (hi - lo)) wide rows.
    Rows of a head share its gate, so ties are broken by (head, row) order.
    Returns uint8 [H][d_k].
    """
    ell = mean_log_retention(gates)
    H = ell.shape[0]
    units = [(ell[h], h, i) for h in range(H) for i in range(d_k)]
    units.sort(key=lambda u: (-u[0], u[1], u[2]))
    n_hi = int(math.floor(len(units) * (budget - lo) / (hi - lo) + 1e-9))
    bits = np.full((H, d_k), lo, np.uint8)
    for _, h, i in units[:n_hi]:
        bits[h, i] = hi
    return bits


# ---------------------------------------------------------------------------
# storage accounting (Appendix D; Appendix F.3 Eq. serving_capacity)
def compact_bits_qwen(budget: float, n_heads: int = 2304, n_pivots: int = 32, dk: int = 128,
                      dv: int = 128, scale_bits: int = 16) -> float:
    """Eq. compact_qwen: b + scale vectors + pivots replacing 8-bit heads."""
    return budget + scale_bits / dv + scale_bits / dk + (n_pivots / n_heads) * (16 - 8)


def compact_bits_kda(budget: float, n_rows: int = 81920, n_pivot_rows: int = 512, dk: int = 128,
                     dv: int = 128, scale_bits: int = 16) -> float:
    """Eq. compact_kda: b + 0.25 (scale vectors) + 512 FP16 pivot rows."""
    return budget + scale_bits / dv + scale_bits / dk + (n_pivot_rows / n_rows) * (16 - 8)


def packed_bytes_qwen6(layers=48, heads=48, dk=128, dv=128, pivots=32, pivot_scale_slots=False) -> int:
    """Packed Qwen@6 recurrent-state bytes per request (Appendix F.1):
    6-bit codes over all elements with the pivot heads' 8-bit share removed,
    FP16 pivot heads, and FP16 row/column vectors for the integer heads
    (or for every head when pivot scale slots are reserved, Appendix F.3)."""
    per_head = dk * dv
    N = layers * heads * per_head
    code_bits = 6 * N - 8 * pivots * per_head
    pivot_bytes = pivots * per_head * 2
    scale_heads = layers * heads if pivot_scale_slots else layers * heads - pivots
    scale_bytes = scale_heads * (dk + dv) * 2
    assert code_bits % 8 == 0
    return code_bits // 8 + pivot_bytes + scale_bytes


def serving_memory(B: int, L: int, W: int, S: int, K: int, r: int = 5) -> int:
    """M(B, L) = W + (r B + 1) S + B L K  (Eq. serving_capacity)."""
    return W + (r * B + 1) * S + B * L * K
