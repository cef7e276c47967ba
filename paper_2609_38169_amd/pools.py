"""Build state pools for the synthetic serving workloads through the product
path: seeded draws -> CPU setup (libstepq's scale fit and bit allocation)
-> GPU quantize-and-pack (stepq_pool_load)."""
from __future__ import annotations

import numpy as np
import torch

from . import stepq
from . import workloads as W


def row_bits(w: W.Workload, layer: int = 0) -> np.ndarray:
    """Precision map [Hv][d_k]: the lifetime-ranked setup step for the
    lifetime48 workload, the seeded draw otherwise."""
    if w.bits == "lifetime48":
        return stepq.stepq_setup_lifetime_bits(W.calibration_gates(w, layer), w.d_k, budget=6.0, lo=4, hi=8)
    return W.bit_map_draw(w, layer).numpy()


def build_pool(w: W.Workload, layer: int = 0, device="cuda", chunk: int = 128, n_threads: int = 0,
               bits: np.ndarray | None = None, levels: int = stepq.STEPQ_LEVELS_ABSMAX) -> stepq.Pool:
    """Allocate a pool for one layer of ``w`` and fill every slot from its
    seeded initial state.  States are drawn on ``device`` ``chunk`` slots at a
    time, fitted on the host (in the pool's level normalisation) and packed
    on the device."""
    dev = torch.device(device)
    b = row_bits(w, layer) if bits is None else bits
    pool = stepq.Pool(w.n_slots, w.n_v_heads, w.n_qk_heads, w.d_k, w.d_v, b, device=dev, levels=levels)
    for s0 in range(0, w.n_slots, chunk):
        slots = range(s0, min(w.n_slots, s0 + chunk))
        S = W.initial_state(w, layer, slots, device=dev)
        need_bits = np.any(b == 16) or levels != stepq.STEPQ_LEVELS_ABSMAX
        r, c = stepq.stepq_setup_fit(S.cpu(), n_threads=n_threads,
                                     row_bits=np.broadcast_to(b, (len(slots),) + b.shape) if need_bits else None,
                                     levels=levels)
        ids = torch.arange(slots.start, slots.stop, dtype=torch.int32, device=dev)
        pool.load(ids, S, torch.from_numpy(r).to(dev), torch.from_numpy(c).to(dev))
        del S
    torch.cuda.synchronize(dev)
    return pool
