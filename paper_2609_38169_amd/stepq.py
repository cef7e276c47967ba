"""Python binding of libstepq (include/stepq.h).

Argument marshalling only: every function here checks that the tensors it is
handed have the shapes, dtypes and devices the C call assumes (the C ABI
takes bare pointers, so this is the last place a size mismatch can be
caught before a kernel reads out of bounds), then forwards their device
pointers and torch's current HIP stream.  All computation happens in the
library's kernels; there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np
import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
# STEPQ_LIB may name another build of the same library (e.g. a tuning variant)
LIB_PATH = os.environ.get("STEPQ_LIB") or os.path.join(_HERE, "libstepq.so")

STEPQ_F32, STEPQ_BF16 = 0, 1
STEPQ_LEVELS_ABSMAX, STEPQ_LEVELS_POW2 = 0, 1     # N1: z = q / q_b;  N2: z = 2^(8-b) q
STEPQ_STEP_KDA_GATE, STEPQ_STEP_REFIT, STEPQ_STEP_ROW_ABSMAX, STEPQ_STEP_ADJACENT_SLOTS = 1, 2, 4, 8
_STATUS = {0: "STEPQ_OK", 1: "STEPQ_E_INVALID", 2: "STEPQ_E_UNSUPPORTED", 3: "STEPQ_E_NOMEM", 4: "STEPQ_E_HIP"}

EXPORTED = (
    "stepq_pool_bytes", "stepq_pool_plan", "stepq_pool_create", "stepq_pool_destroy", "stepq_pool_device_ptr",
    "stepq_pool_load", "stepq_decode_step", "stepq_decode_step_kda", "stepq_decode_step_ex",
    "stepq_decode_stream_ref",
    "stepq_pool_set_row_weight", "stepq_pool_dequant", "stepq_pool_export", "stepq_pool_import",
    "stepq_pool_export_pivots", "stepq_pool_import_pivots", "stepq_last_error", "stepq_setup_fit",
    "stepq_setup_fit_ex", "stepq_setup_fit_levels", "stepq_setup_lifetime_bits", "stepq_setup_row_impact", "stepq_setup_distortion",
    "stepq_setup_lifetime_weights", "stepq_setup_allocate", "stepq_setup_select_pivots",
    "stepq_setup_mean_log_retention", "stepq_setup_lifetime_costs", "stepq_setup_pivot_risk",
)


class StepqError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{_STATUS.get(status, status)}: {msg}")
        self.status = status


class stepq_launch_desc(ctypes.Structure):
    _fields_ = [("body", ctypes.c_int32), ("first", ctypes.c_int32), ("n_heads", ctypes.c_int32)]


class stepq_pool_desc(ctypes.Structure):
    _fields_ = [("n_slots", ctypes.c_int32), ("n_v_heads", ctypes.c_int32), ("n_qk_heads", ctypes.c_int32),
                ("d_k", ctypes.c_int32), ("d_v", ctypes.c_int32), ("row_bits", ctypes.c_void_p),
                ("levels", ctypes.c_int32)]


_lib = None


def lib():
    """The loaded library.  Raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with paper_2609_38169_amd.build.build()")
        L = ctypes.CDLL(LIB_PATH)
        P, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
        st = ctypes.c_int
        sig = {
            "stepq_pool_bytes": ([P, P, P], st),
            "stepq_pool_plan": ([P, ctypes.c_uint32, P, i32, P, P], st),
            "stepq_pool_create": ([P, P, ctypes.c_size_t, P], st),
            "stepq_pool_destroy": ([P], None),
            "stepq_pool_device_ptr": ([P], P),
            "stepq_pool_load": ([P, P, i32, P, P, P, P], st),
            "stepq_decode_step": ([P, P, i32, P, P, P, P, P, st, P, P], st),
            "stepq_decode_step_kda": ([P, P, i32, P, P, P, P, P, st, P, P], st),
            "stepq_decode_step_ex": ([P, P, i32, P, P, P, P, P, st, ctypes.c_uint32, P, P], st),
            "stepq_decode_stream_ref": ([P, P, i32, P, P, P, P, P, st, ctypes.c_uint32, P, P], st),
            "stepq_pool_set_row_weight": ([P, P, P], st),
            "stepq_pool_dequant": ([P, P, i32, P, P], st),
            "stepq_pool_export": ([P, P, i32, P, P, P, P], st),
            "stepq_pool_import": ([P, P, i32, P, P, P, P], st),
            "stepq_pool_export_pivots": ([P, P, i32, P, P], st),
            "stepq_pool_import_pivots": ([P, P, i32, P, P], st),
            "stepq_setup_fit_ex": ([i64, i32, i32, P, P, P, P, P, i32], st),
            "stepq_setup_fit_levels": ([i64, i32, i32, P, P, P, i32, P, P, i32], st),
            "stepq_setup_row_impact": ([i64, i32, i32, P, P, P, P, i32, ctypes.c_double, P, P], st),
            "stepq_setup_distortion": ([i64, i32, i32, i32, P, P, P, i32, P, i32, P, i32], st),
            "stepq_setup_lifetime_weights": ([i32, P, i32, P], st),
            "stepq_setup_mean_log_retention": ([i64, i32, i32, P, i32, i32, P], st),
            "stepq_setup_lifetime_costs": ([i32, i32, P, P, i32, P], st),
            "stepq_setup_pivot_risk": ([i32, P, P, i32, i32, i32, P], st),
            "stepq_setup_allocate": ([i32, i32, P, P, P, ctypes.c_double, i32, P], st),
            "stepq_setup_select_pivots": ([i32, P, i32, P], st),
            "stepq_last_error": ([], ctypes.c_char_p),
            "stepq_setup_fit": ([i64, i32, i32, P, P, P, P, i32], st),
            "stepq_setup_lifetime_bits": ([P, i32, i32, i32, i32, ctypes.c_double, i32, i32, P], st),
        }
        for name, (args, res) in sig.items():
            fn = getattr(L, name)
            fn.argtypes = args
            fn.restype = res
        _lib = L
    return _lib


def _check(status: int):
    if status != 0:
        raise StepqError(status, lib().stepq_last_error().decode())


def _stream(stream):
    if stream is None:
        return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    if isinstance(stream, torch.cuda.Stream):
        return ctypes.c_void_p(stream.cuda_stream)
    return ctypes.c_void_p(int(stream))


def _dev(t: torch.Tensor, name: str, dtype, shape, device):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.device != device:
        raise ValueError(f"{name} is on {t.device}, the pool is on {device}")
    if t.dtype != dtype:
        raise TypeError(f"{name} has dtype {t.dtype}, expected {dtype}")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def _desc(n_slots, n_v_heads, n_qk_heads, d_k, d_v, row_bits: np.ndarray, levels: int = STEPQ_LEVELS_ABSMAX):
    bits = np.ascontiguousarray(row_bits, dtype=np.uint8)
    if bits.shape != (n_v_heads, d_k):
        raise ValueError(f"row_bits has shape {bits.shape}, expected {(n_v_heads, d_k)}")
    d = stepq_pool_desc(n_slots, n_v_heads, n_qk_heads, d_k, d_v, bits.ctypes.data_as(ctypes.c_void_p), int(levels))
    return d, bits


# ---------------------------------------------------------------------------
# C-ABI functions under their own names
def stepq_pool_bytes(n_slots, n_v_heads, n_qk_heads, d_k, d_v, row_bits, levels=STEPQ_LEVELS_ABSMAX):
    d, _keep = _desc(n_slots, n_v_heads, n_qk_heads, d_k, d_v, row_bits, levels)
    pb, sb = ctypes.c_size_t(), ctypes.c_size_t()
    _check(lib().stepq_pool_bytes(ctypes.byref(d), ctypes.byref(pb), ctypes.byref(sb)))
    return pb.value, sb.value


def stepq_pool_plan(n_slots, n_v_heads, n_qk_heads, d_k, d_v, row_bits, levels=STEPQ_LEVELS_ABSMAX, flags: int = 0):
    """The launches of one decode step (host only): a list of (body,
    first, n_heads) and the head order [n_v_heads] their head lists index."""
    d, _keep = _desc(n_slots, n_v_heads, n_qk_heads, d_k, d_v, row_bits, levels)
    n = ctypes.c_int32()
    order = np.empty(n_v_heads, np.int32)
    _check(lib().stepq_pool_plan(ctypes.byref(d), int(flags), None, 0, ctypes.byref(n), None))
    buf = (stepq_launch_desc * max(1, n.value))()
    _check(lib().stepq_pool_plan(ctypes.byref(d), int(flags), buf, n.value, ctypes.byref(n),
                                 order.ctypes.data_as(ctypes.c_void_p)))
    return [(x.body, x.first, x.n_heads) for x in buf[:n.value]], order


class Pool:
    """A state pool whose memory is a torch uint8 tensor on the current device."""

    def __init__(self, n_slots, n_v_heads, n_qk_heads, d_k, d_v, row_bits, device=None,
                 levels=STEPQ_LEVELS_ABSMAX):
        self.device = torch.device("cuda", torch.cuda.current_device()) if device is None else torch.device(device)
        self.n_slots, self.Hv, self.Hqk, self.dk, self.dv = n_slots, n_v_heads, n_qk_heads, d_k, d_v
        self.levels = int(levels)
        self.row_bits = np.ascontiguousarray(row_bits, dtype=np.uint8).copy()
        self.pool_bytes, self.slot_bytes = stepq_pool_bytes(n_slots, n_v_heads, n_qk_heads, d_k, d_v, self.row_bits,
                                                            self.levels)
        with torch.cuda.device(self.device):
            self.memory = torch.empty(self.pool_bytes, dtype=torch.uint8, device=self.device)
            if self.memory.data_ptr() % 256:
                raise RuntimeError("torch returned pool memory that is not 256-byte aligned")
            d, _keep = _desc(n_slots, n_v_heads, n_qk_heads, d_k, d_v, self.row_bits, self.levels)
            h = ctypes.c_void_p()
            _check(lib().stepq_pool_create(ctypes.byref(d), ctypes.c_void_p(self.memory.data_ptr()),
                                           self.pool_bytes, ctypes.byref(h)))
        self.handle = h

    def close(self):
        if getattr(self, "handle", None):
            with torch.cuda.device(self.device):
                lib().stepq_pool_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # convenience forms of the calls below
    def load(self, slot_ids, state, r, c, stream=None):
        stepq_pool_load(self, slot_ids, state, r, c, stream)

    # refit: False (frozen scales), True (dual-axis refit) or "row_absmax"
    # (the single-axis INT-b baseline); adjacent: the STEPQ_STEP_ADJACENT_SLOTS
    # hint (slot_ids[b] = slot_ids[0] + b)
    def step(self, slot_ids, q, k, v, alpha, beta, o, stream=None, refit=False, adjacent=False):
        flags = _refit_flags(refit) | (STEPQ_STEP_ADJACENT_SLOTS if adjacent else 0)
        if flags:
            stepq_decode_step_ex(self, slot_ids, q, k, v, alpha, beta, o, flags, stream)
        else:
            stepq_decode_step(self, slot_ids, q, k, v, alpha, beta, o, stream)

    def step_kda(self, slot_ids, q, k, v, gate, beta, o, stream=None, refit=False, adjacent=False):
        flags = _refit_flags(refit) | (STEPQ_STEP_ADJACENT_SLOTS if adjacent else 0)
        if flags:
            stepq_decode_step_ex(self, slot_ids, q, k, v, gate, beta, o, STEPQ_STEP_KDA_GATE | flags, stream)
        else:
            stepq_decode_step_kda(self, slot_ids, q, k, v, gate, beta, o, stream)

    def set_row_weight(self, w, stream=None):
        stepq_pool_set_row_weight(self, w, stream)

    def prepare_step(self, slot_ids, q, k, v, alpha, beta, o, stream=None, refit=False, adjacent=False):
        """Validate the arguments of one decode step once and return a
        callable that launches it with the cached pointers (for decode loops
        where the per-call checks would dominate the launch cost).  alpha of
        shape [B][Hv][d_k] selects the channel-wise (KDA) gate; refit the
        online scale refit; adjacent the STEPQ_STEP_ADJACENT_SLOTS hint."""
        kda = alpha.dim() == 3
        args = _step_args(self, slot_ids, q, k, v, alpha, beta, o, stream, kda)
        keep = (slot_ids, q, k, v, alpha, beta, o)      # the tensors must outlive the callable
        if refit or adjacent:
            flags = ctypes.c_uint32(_refit_flags(refit) | (STEPQ_STEP_KDA_GATE if kda else 0) |
                                    (STEPQ_STEP_ADJACENT_SLOTS if adjacent else 0))
            fn = lib().stepq_decode_step_ex
            args = args[:9] + (flags,) + args[9:]
        else:
            fn = lib().stepq_decode_step_kda if kda else lib().stepq_decode_step

        def launch():
            _ = keep
            st = fn(*args)
            if st != 0:
                _check(st)
        return launch

    def prepare_stream_ref(self, slot_ids, q, k, v, alpha, beta, o, stream=None, adjacent=False):
        """prepare_step for the memory-only reference of a decode step
        (stepq_decode_stream_ref): same tiles, order and traffic, no
        arithmetic; o receives zeros."""
        args = _step_args(self, slot_ids, q, k, v, alpha, beta, o, stream, False)
        keep = (slot_ids, q, k, v, alpha, beta, o)
        flags = ctypes.c_uint32(STEPQ_STEP_ADJACENT_SLOTS if adjacent else 0)
        args = args[:9] + (flags,) + args[9:]
        fn = lib().stepq_decode_stream_ref

        def launch():
            _ = keep
            st = fn(*args)
            if st != 0:
                _check(st)
        return launch

    def dequant(self, slot_ids, out, stream=None):
        stepq_pool_dequant(self, slot_ids, out, stream)

    def export(self, slot_ids, codes, r, c, stream=None):
        stepq_pool_export(self, slot_ids, codes, r, c, stream)

    def import_(self, slot_ids, codes, r, c, stream=None):
        stepq_pool_import(self, slot_ids, codes, r, c, stream)

    def export_pivots(self, slot_ids, pivots, stream=None):
        stepq_pool_export_pivots(self, slot_ids, pivots, stream)

    def import_pivots(self, slot_ids, pivots, stream=None):
        stepq_pool_import_pivots(self, slot_ids, pivots, stream)


def stepq_pool_create(n_slots, n_v_heads, n_qk_heads, d_k, d_v, row_bits, device=None) -> Pool:
    return Pool(n_slots, n_v_heads, n_qk_heads, d_k, d_v, row_bits, device)


def stepq_pool_destroy(pool: Pool):
    pool.close()


def stepq_pool_device_ptr(pool: Pool) -> int:
    return lib().stepq_pool_device_ptr(pool.handle)


def _ids(pool: Pool, slot_ids: torch.Tensor):
    if slot_ids.dim() != 1:
        raise ValueError("slot_ids must be 1-D")
    n = slot_ids.shape[0]
    return n, _dev(slot_ids, "slot_ids", torch.int32, (n,), pool.device)


def stepq_pool_load(pool: Pool, slot_ids, state, r, c, stream=None):
    n, ids = _ids(pool, slot_ids)
    P = pool
    _check(lib().stepq_pool_load(
        pool.handle, ids, n,
        _dev(state, "state", torch.float32, (n, P.Hv, P.dk, P.dv), P.device),
        _dev(r, "r", torch.float32, (n, P.Hv, P.dk), P.device),
        _dev(c, "c", torch.float32, (n, P.Hv, P.dv), P.device), _stream(stream)))


def _refit_flags(refit) -> int:
    if refit is False:
        return 0
    if refit is True:
        return STEPQ_STEP_REFIT
    if refit == "row_absmax":
        return STEPQ_STEP_ROW_ABSMAX
    raise ValueError(f"refit must be False, True or 'row_absmax', not {refit!r}")


def _step_args(pool: Pool, slot_ids, q, k, v, gate, beta, o, stream, kda: bool):
    """Checked pointer arguments of a decode-step call, in C order without
    the flags: (pool, ids, batch, q, k, v, gate, beta, dtype, o, stream)."""
    n, ids = _ids(pool, slot_ids)
    P = pool
    dt = q.dtype
    if dt not in (torch.float32, torch.bfloat16):
        raise TypeError("activations must be float32 or bfloat16")
    code = STEPQ_F32 if dt == torch.float32 else STEPQ_BF16
    gshape = (n, P.Hv, P.dk) if kda else (n, P.Hv)
    return (pool.handle, ids, n,
            _dev(q, "q", dt, (n, P.Hqk, P.dk), P.device),
            _dev(k, "k", dt, (n, P.Hqk, P.dk), P.device),
            _dev(v, "v", dt, (n, P.Hv, P.dv), P.device),
            _dev(gate, "gate" if kda else "alpha", dt, gshape, P.device),
            _dev(beta, "beta", dt, (n, P.Hv), P.device), code,
            _dev(o, "o", torch.float32, (n, P.Hv, P.dv), P.device), _stream(stream))


def stepq_decode_step(pool: Pool, slot_ids, q, k, v, alpha, beta, o, stream=None):
    _check(lib().stepq_decode_step(*_step_args(pool, slot_ids, q, k, v, alpha, beta, o, stream, False)))


def stepq_decode_step_kda(pool: Pool, slot_ids, q, k, v, gate, beta, o, stream=None):
    _check(lib().stepq_decode_step_kda(*_step_args(pool, slot_ids, q, k, v, gate, beta, o, stream, True)))


def stepq_decode_step_ex(pool: Pool, slot_ids, q, k, v, gate, beta, o, flags: int, stream=None):
    a = _step_args(pool, slot_ids, q, k, v, gate, beta, o, stream, bool(flags & STEPQ_STEP_KDA_GATE))
    _check(lib().stepq_decode_step_ex(*a[:9], ctypes.c_uint32(flags), *a[9:]))


def stepq_pool_set_row_weight(pool: Pool, w, stream=None):
    """w: [Hv][d_k] row-impact factors (host array or tensor), logical row
    order; uploaded in order on the stream (torch's current one by default)."""
    wt = np.ascontiguousarray(w.cpu().numpy() if isinstance(w, torch.Tensor) else w, dtype=np.float32)
    if wt.shape != (pool.Hv, pool.dk):
        raise ValueError(f"row weights have shape {wt.shape}, expected {(pool.Hv, pool.dk)}")
    with torch.cuda.device(pool.device):
        _check(lib().stepq_pool_set_row_weight(pool.handle, wt.ctypes.data_as(ctypes.c_void_p), _stream(stream)))


def stepq_pool_dequant(pool: Pool, slot_ids, out, stream=None):
    n, ids = _ids(pool, slot_ids)
    P = pool
    _check(lib().stepq_pool_dequant(pool.handle, ids, n,
                                    _dev(out, "out", torch.float32, (n, P.Hv, P.dk, P.dv), P.device),
                                    _stream(stream)))


def stepq_pool_export(pool: Pool, slot_ids, codes, r, c, stream=None):
    n, ids = _ids(pool, slot_ids)
    P = pool
    _check(lib().stepq_pool_export(
        pool.handle, ids, n,
        _dev(codes, "codes", torch.int8, (n, P.Hv, P.dk, P.dv), P.device),
        _dev(r, "r", torch.float32, (n, P.Hv, P.dk), P.device),
        _dev(c, "c", torch.float32, (n, P.Hv, P.dv), P.device), _stream(stream)))


def stepq_pool_import(pool: Pool, slot_ids, codes, r, c, stream=None):
    n, ids = _ids(pool, slot_ids)
    P = pool
    _check(lib().stepq_pool_import(
        pool.handle, ids, n,
        _dev(codes, "codes", torch.int8, (n, P.Hv, P.dk, P.dv), P.device),
        _dev(r, "r", torch.float32, (n, P.Hv, P.dk), P.device),
        _dev(c, "c", torch.float32, (n, P.Hv, P.dv), P.device), _stream(stream)))


def stepq_pool_export_pivots(pool: Pool, slot_ids, pivots, stream=None):
    """pivots: [n][Hv][d_k][d_v] torch.int16 or uint16 on the pool's device
    (binary16 bit patterns of the pivot rows, zeros elsewhere)."""
    n, ids = _ids(pool, slot_ids)
    P = pool
    _check(lib().stepq_pool_export_pivots(pool.handle, ids, n,
                                          _dev16(pivots, "pivots", (n, P.Hv, P.dk, P.dv), P.device), _stream(stream)))


def stepq_pool_import_pivots(pool: Pool, slot_ids, pivots, stream=None):
    n, ids = _ids(pool, slot_ids)
    P = pool
    _check(lib().stepq_pool_import_pivots(pool.handle, ids, n,
                                          _dev16(pivots, "pivots", (n, P.Hv, P.dk, P.dv), P.device), _stream(stream)))


def _dev16(t, name, shape, device):
    # binary16 bit patterns travel in a 16-bit integer tensor
    if not isinstance(t, torch.Tensor) or t.dtype not in (torch.int16, torch.uint16):
        raise TypeError(f"{name} must be a torch.int16 or torch.uint16 tensor of binary16 bit patterns")
    return _dev(t, name, t.dtype, shape, device)


def stepq_last_error() -> str:
    return lib().stepq_last_error().decode()


# ---------------------------------------------------------------------------
# CPU setup step (host arrays)
def stepq_setup_fit(state, row_weight=None, n_threads: int = 0, row_bits=None, levels=STEPQ_LEVELS_ABSMAX):
    """state: [..., d_k, d_v] float32 (host) -> (r [..., d_k], c [..., d_v]) float32 numpy.
    row_bits [..., d_k] (optional under N1, needed under N2): pivot rows (16)
    are left out of c; levels: the pool's level normalisation."""
    S = np.ascontiguousarray(state.numpy() if isinstance(state, torch.Tensor) else state, dtype=np.float32)
    dk, dv = S.shape[-2:]
    lead = S.shape[:-2]
    n = int(np.prod(lead)) if lead else 1
    r = np.empty(lead + (dk,), np.float32)
    c = np.empty(lead + (dv,), np.float32)
    w = None
    if row_weight is not None:
        w = np.ascontiguousarray(np.broadcast_to(row_weight, lead + (dk,)), dtype=np.float32)
    vp = lambda a: None if a is None else a.ctypes.data_as(ctypes.c_void_p)
    if levels != STEPQ_LEVELS_ABSMAX:
        if row_bits is None:
            raise ValueError("the N2 fit needs the row widths")
        b = np.ascontiguousarray(np.broadcast_to(row_bits, lead + (dk,)), dtype=np.uint8)
        _check(lib().stepq_setup_fit_levels(n, dk, dv, vp(S), vp(w), vp(b), int(levels), vp(r), vp(c), n_threads))
    elif row_bits is None:
        _check(lib().stepq_setup_fit(n, dk, dv, vp(S), vp(w), vp(r), vp(c), n_threads))
    else:
        b = np.ascontiguousarray(np.broadcast_to(row_bits, lead + (dk,)), dtype=np.uint8)
        _check(lib().stepq_setup_fit_ex(n, dk, dv, vp(S), vp(w), vp(b), vp(r), vp(c), n_threads))
    return r, c


def stepq_setup_lifetime_bits(gates, d_k: int, budget: float = 6.0, lo: int = 4, hi: int = 8):
    """gates [T][B][H] (host) -> row_bits uint8 [H][d_k]."""
    g = np.ascontiguousarray(gates.numpy() if isinstance(gates, torch.Tensor) else gates, dtype=np.float64)
    T, B, H = g.shape
    out = np.empty((H, d_k), np.uint8)
    st = lib().stepq_setup_lifetime_bits(g.ctypes.data_as(ctypes.c_void_p), T, B, H, d_k, budget, lo, hi,
                                         out.ctypes.data_as(ctypes.c_void_p))
    if st != 0:
        raise StepqError(st, "invalid lifetime allocation arguments")
    return out


# ---------------------------------------------------------------------------
# calibration side of the setup step (host arrays)
def _vp(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _host(a, dtype):
    return np.ascontiguousarray(a.cpu().numpy() if isinstance(a, torch.Tensor) else a, dtype=dtype)


def _setup_check(st, what):
    if st != 0:
        raise StepqError(st, what)


def stepq_setup_row_impact(q, k, beta, gate, gamma: float = 0.25):
    """q, k [T][H][d_k], beta [T][H], gate [T][H] or [T][H][d_k] -> (w, omega) [H][d_k]."""
    q, k = _host(q, np.float32), _host(k, np.float32)
    beta, gate = _host(beta, np.float32), _host(gate, np.float32)
    T, H, dk = q.shape
    w = np.empty((H, dk), np.float32)
    om = np.empty((H, dk), np.float64)
    _setup_check(lib().stepq_setup_row_impact(T, H, dk, _vp(q), _vp(k), _vp(beta), _vp(gate), int(gate.ndim == 3),
                                              float(gamma), _vp(w), _vp(om)), "row impact")
    return w, om


def stepq_setup_distortion(states, cand_bits, unit: str, row_weight=None, pivots=None, n_threads: int = 0):
    """states [C][H][d_k][d_v] -> d [U][len(cand_bits)] (unit "row" or "head")."""
    S = _host(states, np.float32)
    C, H, dk, dv = S.shape
    cb = np.ascontiguousarray(cand_bits, dtype=np.int32)
    w = None if row_weight is None else _host(row_weight, np.float32)
    pv = None if pivots is None else _host(pivots, np.uint8)
    u = {"row": 0, "head": 1}[unit]
    out = np.empty((H * dk if u == 0 else H, len(cb)), np.float64)
    _setup_check(lib().stepq_setup_distortion(C, H, dk, dv, _vp(S), _vp(w), _vp(pv), len(cb), _vp(cb), u, _vp(out),
                                              n_threads), "distortion")
    return out


def stepq_setup_lifetime_weights(ell, horizon: int):
    e = _host(ell, np.float64)
    out = np.empty(e.shape, np.float64)
    _setup_check(lib().stepq_setup_lifetime_weights(e.size, _vp(e), horizon, _vp(out)), "lifetime weights")
    return out


def stepq_setup_mean_log_retention(gates, d_k: int, unit: str):
    """ell per unit (Appendix A.3) from calibration gates [T][H] (scalar,
    GDN) or [T][H][d_k] (channel-wise, KDA): [H * d_k] for unit "row",
    [H] for unit "head"."""
    g = _host(gates, np.float32)
    if g.ndim not in (2, 3) or (g.ndim == 3 and g.shape[2] != d_k):
        raise ValueError("gates must be [T][H] or [T][H][d_k]")
    T, H = g.shape[:2]
    u = {"row": 0, "head": 1}[unit]
    out = np.empty(H * d_k if u == 0 else H, np.float64)
    _setup_check(lib().stepq_setup_mean_log_retention(T, H, d_k, _vp(g), int(g.ndim == 3), u, _vp(out)),
                 "mean log retention")
    return out


def stepq_setup_lifetime_costs(L, d, n_cand: int):
    """cost [U][n_cand] = L_u d_u(b) over the first n_cand columns of d [U][*]."""
    Lh, dh = _host(L, np.float64), _host(d, np.float64)
    U, stride = dh.shape
    out = np.empty((U, n_cand), np.float64)
    _setup_check(lib().stepq_setup_lifetime_costs(U, n_cand, _vp(Lh), _vp(dh), stride, _vp(out)), "lifetime costs")
    return out


def stepq_setup_pivot_risk(L, d, col_int: int, col_f16: int):
    """risk_u = L_u (d_u[col_int] - d_u[col_f16]) for d [U][*]."""
    Lh, dh = _host(L, np.float64), _host(d, np.float64)
    U, stride = dh.shape
    out = np.empty(U, np.float64)
    _setup_check(lib().stepq_setup_pivot_risk(U, _vp(Lh), _vp(dh), stride, col_int, col_f16, _vp(out)), "pivot risk")
    return out


def stepq_setup_allocate(cost, n_u, cand_bits, budget: float, method: str = "dp"):
    """cost [U][n_cand], n_u [U] -> candidate index per unit (method "dp" or "lagrangian")."""
    c = _host(cost, np.float64)
    U, nc = c.shape
    n = np.ascontiguousarray(np.broadcast_to(n_u, (U,)), dtype=np.int32)
    cb = np.ascontiguousarray(cand_bits, dtype=np.int32)
    out = np.empty(U, np.int32)
    _setup_check(lib().stepq_setup_allocate(U, nc, _vp(cb), _vp(c), _vp(n), float(budget),
                                            {"dp": 0, "lagrangian": 1}[method], _vp(out)), "allocation")
    return out


def stepq_setup_select_pivots(risk, count: int):
    r = _host(risk, np.float64)
    out = np.empty(r.shape, np.uint8)
    _setup_check(lib().stepq_setup_select_pivots(r.size, _vp(r), count, _vp(out)), "pivot selection")
    return out.astype(bool)
