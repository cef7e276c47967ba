"""GPU parity at the extremes of the decode step, lockstep against the fp64
oracle through the C ABI: every slot of the 2048-slot pool stepped in one
launch (65,536 workgroups), and the degenerate gates of the update:
alpha = 0 (the state is replaced by the rank-one write beta k v^T),
beta = 0 (pure decay, X = alpha S), and channel-wise gates of exactly 0 or 1
(rows forgotten or kept whole)."""
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
