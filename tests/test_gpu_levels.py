"""GPU parity under the second level normalisation N2 (a b-bit code q stands
for the level 2^(8-b) q, the paper's KDA codebook; Appendix C.1), against
the fp64 oracle through the C ABI: the boundary pack and reconstruction,
and the pool-sized decode step in all three scale modes, with the scalar
GDN gate and with KDA's channel-wise gate."""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_38169_amd import stepq, workloads as W
from paper_2609_38169_amd.pools import row_bits
import _parity as PT

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda", 0)
N2 = stepq.STEPQ_LEVELS_POW2


def _say(*a):
    print(*a, flush=True)


@pytest.mark.parametrize("idx", [0, 3])
def test_pow2_pool_load_and_dequant(idx):
    """stepq_pool_load quantizes with the N2 levels (the oracle's quantizer on
    the same scales, which the host fit and the oracle's fit agree on bit for
    bit), and stepq_pool_dequant reconstructs r c 2^(8-b) q to well inside
    one level."""
    w = W.workload(idx)
    n = min(w.n_slots, 8)
    _say(f"N2 pool_load {w.name}: {n} slots")
    bits = row_bits(w)
    S = W.initial_state(w, 0, range(n), device=DEV)
    tb = np.broadcast_to(bits[None], (n,) + bits.shape)
    r, c = stepq.stepq_setup_fit(S.cpu(), row_bits=tb, levels=N2)
    Sn = S.cpu().numpy().reshape(-1, w.d_k, w.d_v)
    ro, co = oracle.fit_absmax(Sn, bits=tb.reshape(-1, w.d_k), levels=oracle.LEVELS_POW2)
    assert np.array_equal(r.reshape(ro.shape), ro) and np.array_equal(c.reshape(co.shape), co)
    pool = stepq.Pool(n, w.n_v_heads, w.n_qk_heads, w.d_k, w.d_v, bits, device=DEV, levels=N2)
    ids = torch.arange(n, dtype=torch.int32, device=DEV)
    pool.load(ids, S, torch.from_numpy(r).to(DEV), torch.from_numpy(c).to(DEV))
    codes = torch.empty((n, w.n_v_heads, w.d_k, w.d_v), dtype=torch.int8, device=DEV)
    pool.export(ids, codes, torch.empty((n, w.n_v_heads, w.d_k), device=DEV),
                torch.empty((n, w.n_v_heads, w.d_v), device=DEV))
    deq = torch.empty((n, w.n_v_heads, w.d_k, w.d_v), dtype=torch.float32, device=DEV)
    pool.dequant(ids, deq)
    torch.cuda.synchronize()
    oc, y = oracle.quantize(Sn.astype(np.float64), ro, co, tb.reshape(-1, w.d_k), want_y=True,
                            levels=oracle.LEVELS_POW2)
    got = codes.cpu().numpy().reshape(oc.shape)
    PT.compare_codes(got, oc, y, "N2 pool_load codes")
    ref = oracle.dequant(got, ro, co, tb.reshape(-1, w.d_k), levels=oracle.LEVELS_POW2)
    step = ro.astype(np.float64)[:, :, None] * co.astype(np.float64)[:, None, :] * \
        (2.0 ** (8 - tb.reshape(-1, w.d_k).astype(np.int64)))[:, :, None]
    assert np.all(np.abs(deq.cpu().numpy().reshape(ref.shape) - ref) <= 1e-3 * step)


@pytest.mark.parametrize("mode", [False, True, "row_absmax"])
def test_pow2_pool_b512_lockstep(mode):
    """The B=512 pool under N2, all slots stepped, sampled slots lockstep."""
    w = W.workload(2)
    PT.lockstep_run(w, 6, np.array([0, 131, 511]), DEV, refit=mode, say=_say, levels=N2)


@pytest.mark.parametrize("mode", [False, True])
def test_pow2_kda_lockstep(mode):
    """KDA's channel-wise gates with its own code normalisation (the paper's
    KDA configuration), on the B=512 pool."""
    w = W.workload(2)
    PT.lockstep_run(w, 4, np.array([3, 256, 510]), DEV, refit=mode, kda=True, say=_say, levels=N2)


def test_pow2_pivots_and_fp16_heads():
    """N2 with FP16 pivot rows and whole FP16 heads (which carry no levels)."""
    w = W.workload(2)
    bits = row_bits(w)
    bits[W.pivot_mask_draw(w).numpy()] = 16
    bits[W.pivot_head_draw(w, 0, 1).numpy()] = 16
    PT.lockstep_run(w, 3, np.array([0, 400]), DEV, refit=True, say=_say, bits=bits, levels=N2)
