"""Seeded synthetic workloads for the quantized gated-Delta decode step.

This module only draws random numbers with the shapes and value
distributions of the serving workloads; it holds none of the method's
arithmetic (no scale fitting, no bit allocation, no quantization, no
update).  Both the HIP path and the fp64 oracle consume what it returns.

Every draw is keyed by (config, layer, step, stream) through its own
``torch.Generator``, so any single step can be regenerated without the
steps before it.  Values depend on the device the draw is made on (torch's
CPU and GPU generators differ); small configurations draw on the CPU, the
pool-sized ones on the GPU.

Workload shapes (paper: GDN/KDA recurrent layers with d_k = d_v = 128 and
32-48 state heads per layer, Appendix D and Table C1; batch sizes up to 512
concurrent requests, Appendix F):

  0  tiny       1 request x 4 heads, d=64, 32 steps, fp32 activations,
                i.i.d. {4,8} bit per key row
  1  layer_b64  64 requests x 32 value heads (16 q/k heads), d=128,
                256 steps, fp32 activations, long-lived gates, row widths
                chosen by lifetime ranking (setup step, not here)
  2  pool_b512  2048-slot pool, 512 active requests x 32 heads, d=128,
                128 steps, bf16 activations, 64 rows @8 + 64 rows @4 per head
  3  pool_4bit  512 requests x 32 heads, d=128, 128 steps, bf16,
                64 @2 + 32 @4 + 32 @8 per head, heavy-tailed initial state
  4  stack48    48 layers x 256 requests x 32 value heads (16 q/k), d=128,
                64 steps, bf16, 64 @8 + 64 @4 per head
"""
from __future__ import annotations

import dataclasses

import torch

__all__ = [
    "Workload", "WORKLOADS", "workload",
    "initial_state", "step_inputs", "bit_map_draw", "calibration_gates",
    "active_slots", "rotation_slots",
]


@dataclasses.dataclass(frozen=True)
class Workload:
    index: int
    name: str
    n_slots: int          # state slots in the pool
    batch: int            # active requests per decode step
    n_v_heads: int
    n_qk_heads: int
    d_k: int
    d_v: int
    steps: int
    layers: int
    act_dtype: torch.dtype
    gate: str             # "softplus" (exp(-softplus(N)*0.1)) or "near1" (1-U(0,0.05))
    init: str             # "normal" (N(0, 0.05^2)) or "heavy" (N(0,1)*g_r*g_c, lognormal gains)
    bits: str             # "iid48", "lifetime48", "half48", "mix248"
    calib_steps: int = 32

    @property
    def tiles_per_step(self) -> int:
        return self.batch * self.n_v_heads


WORKLOADS = {
    0: Workload(0, "tiny", 1, 1, 4, 4, 64, 64, 32, 1, torch.float32, "softplus", "normal", "iid48"),
    1: Workload(1, "layer_b64", 64, 64, 32, 16, 128, 128, 256, 1, torch.float32, "near1", "normal", "lifetime48"),
    2: Workload(2, "pool_b512", 2048, 512, 32, 32, 128, 128, 128, 1, torch.bfloat16, "near1", "normal", "half48"),
    3: Workload(3, "pool_4bit", 512, 512, 32, 32, 128, 128, 128, 1, torch.bfloat16, "near1", "heavy", "mix248"),
    4: Workload(4, "stack48", 256, 256, 32, 16, 128, 128, 64, 48, torch.bfloat16, "near1", "normal", "half48"),
}


def workload(index: int) -> Workload:
    return WORKLOADS[int(index)]


# ---------------------------------------------------------------------------
# seeding
_MASK64 = (1 << 64) - 1


def _mix(*parts: int) -> int:
    """splitmix64 over the key parts -> a 63-bit seed."""
    h = 0x9E3779B97F4A7C15
    for p in parts:
        h = (h ^ (int(p) & _MASK64)) & _MASK64
        h = (h + 0x9E3779B97F4A7C15) & _MASK64
        z = h
        z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & _MASK64
        z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & _MASK64
        h = z ^ (z >> 31)
    return h & ((1 << 63) - 1)


_STREAM = {"init": 1, "q": 2, "k": 3, "v": 4, "alpha": 5, "beta": 6,
           "bits": 7, "calib": 8, "slots": 9, "gain_r": 10, "gain_c": 11, "kda": 12,
           "roww": 13, "pivots": 14, "pivot_heads": 15}


def _gen(device, w: Workload, layer: int, step: int, stream: str, chunk: int = 0) -> torch.Generator:
    dev = torch.device(device)
    g = torch.Generator(device=dev)
    g.manual_seed(_mix(w.index, layer, step, _STREAM[stream], chunk))
    return g


# ---------------------------------------------------------------------------
# draws
def initial_state(w: Workload, layer: int = 0, slots: range | None = None,
                  device="cpu") -> torch.Tensor:
    """fp32 initial states [len(slots)][Hv][d_k][d_v] for pool slots ``slots``.

    Each slot is drawn from its own generator, so any subset of the pool can be
    regenerated alone.  "normal": entries N(0, 0.05^2).  "heavy": entries
    N(0,1) * g_r[i] * g_c[j] with per-tile gains exp(N(0,1)) along key rows and
    value columns (two-axis magnitude structure of Section 4.2).
    """
    if slots is None:
        slots = range(w.n_slots)
    shape = (w.n_v_heads, w.d_k, w.d_v)
    out = torch.empty((len(slots),) + shape, dtype=torch.float32, device=device)
    for n, s in enumerate(slots):
        g = _gen(device, w, layer, 0, "init", s)
        x = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
        if w.init == "normal":
            x.mul_(0.05)
        elif w.init == "heavy":
            gr = torch.exp(torch.randn((w.n_v_heads, w.d_k, 1), generator=_gen(device, w, layer, 0, "gain_r", s),
                                       device=device, dtype=torch.float32))
            gc = torch.exp(torch.randn((w.n_v_heads, 1, w.d_v), generator=_gen(device, w, layer, 0, "gain_c", s),
                                       device=device, dtype=torch.float32))
            x.mul_(gr).mul_(gc)
        else:
            raise ValueError(w.init)
        out[n] = x
    return out


def _gates(w: Workload, g: torch.Generator, shape, device) -> torch.Tensor:
    if w.gate == "softplus":
        x = torch.randn(shape, generator=g, device=device, dtype=torch.float64)
        return torch.exp(-torch.nn.functional.softplus(x) * 0.1)
    if w.gate == "near1":
        u = torch.rand(shape, generator=g, device=device, dtype=torch.float64)
        return 1.0 - 0.05 * u
    raise ValueError(w.gate)


def step_inputs(w: Workload, layer: int, step: int, device="cpu") -> dict:
    """Decode-step activations for all ``batch`` requests.

    q, k: [B][Hqk][d_k] drawn N(0,1) then L2-normalised per head (in fp64, then
    cast to the activation dtype, so bf16 keys are only approximately unit);
    v: [B][Hv][d_v] N(0,1); alpha, beta: [B][Hv], beta = sigmoid(N(0,1)),
    alpha per the workload's gate law.
    """
    B, Hq, Hv = w.batch, w.n_qk_heads, w.n_v_heads
    dt = w.act_dtype

    def unit(stream, d):
        x = torch.randn((B, Hq, d), generator=_gen(device, w, layer, step, stream), device=device,
                        dtype=torch.float64)
        return (x / torch.linalg.vector_norm(x, dim=-1, keepdim=True)).to(dt)

    q = unit("q", w.d_k)
    k = unit("k", w.d_k)
    v = torch.randn((B, Hv, w.d_v), generator=_gen(device, w, layer, step, "v"), device=device,
                    dtype=torch.float64).to(dt)
    alpha = _gates(w, _gen(device, w, layer, step, "alpha"), (B, Hv), device).to(dt)
    beta = torch.sigmoid(torch.randn((B, Hv), generator=_gen(device, w, layer, step, "beta"),
                                     device=device, dtype=torch.float64)).to(dt)
    return {"q": q, "k": k, "v": v, "alpha": alpha, "beta": beta}


def kda_gates(w: Workload, layer: int, step: int, device="cpu") -> torch.Tensor:
    """Channel-wise retention gates d_{t,i} for the KDA form of the update,
    [B][Hv][d_k] in the activation dtype: one draw per key row from the
    workload's gate law, on a stream of its own."""
    g = _gen(device, w, layer, step, "kda")
    return _gates(w, g, (w.batch, w.n_v_heads, w.d_k), device).to(w.act_dtype)


def row_weight_draw(w: Workload, layer: int = 0, sigma: float = 0.5) -> torch.Tensor:
    """Synthetic row-impact factors, float32 [Hv][d_k]: lognormal with log
    standard deviation sigma, each head's logs centred so that its geometric
    mean is one (the normalisation the factors carry)."""
    g = _gen("cpu", w, layer, 0, "roww")
    x = torch.randn((w.n_v_heads, w.d_k), generator=g, dtype=torch.float64) * sigma
    return torch.exp(x - x.mean(dim=1, keepdim=True)).to(torch.float32)


def pivot_mask_draw(w: Workload, layer: int = 0, head_frac: float = 0.25, max_rows: int = 3) -> torch.Tensor:
    """Synthetic FP16 pivot rows, bool [Hv][d_k]: a seeded share of the heads
    get 1 .. max_rows pivot rows at seeded positions (the paper keeps a few
    hundred rows of a model in FP16, spread over its heads)."""
    g = _gen("cpu", w, layer, 0, "pivots")
    mask = torch.zeros((w.n_v_heads, w.d_k), dtype=torch.bool)
    pick = torch.rand(w.n_v_heads, generator=g) < head_frac
    count = torch.randint(1, max_rows + 1, (w.n_v_heads,), generator=g)
    for h in range(w.n_v_heads):
        if pick[h]:
            mask[h, torch.randperm(w.d_k, generator=g)[: int(count[h])]] = True
    return mask


def pivot_head_draw(w: Workload, layer: int = 0, count: int = 1) -> torch.Tensor:
    """Synthetic FP16 pivot heads, bool [Hv]: a seeded choice of ``count``
    value heads kept entirely in FP16 (the paper keeps whole heads of its
    GDN model in FP16)."""
    g = _gen("cpu", w, layer, 0, "pivot_heads")
    mask = torch.zeros(w.n_v_heads, dtype=torch.bool)
    mask[torch.randperm(w.n_v_heads, generator=g)[:count]] = True
    return mask


def calibration_gates(w: Workload, layer: int = 0) -> torch.Tensor:
    """Gate draws from a separate calibration stream, [calib_steps][B][Hv] fp64.

    Same law as the decode gates; used by the lifetime-ranked allocation of
    the layer_b64 workload (mean log retention per head).
    """
    g = _gen("cpu", w, layer, 0, "calib")
    return _gates(w, g, (w.calib_steps, w.batch, w.n_v_heads), "cpu")


def bit_map_draw(w: Workload, layer: int = 0) -> torch.Tensor:
    """Per-(head, key row) bit widths, uint8 [Hv][d_k], for the draw-only maps.

    iid48  : each row 4 or 8 with probability 1/2
    half48 : per head a seeded permutation picks 64 rows @8, the rest @4
    mix248 : per head a seeded permutation picks 32 @8, 32 @4, 64 @2
    lifetime48 is not a draw: it is produced by the lifetime-ranked setup step
    from ``calibration_gates``.
    """
    g = _gen("cpu", w, layer, 0, "bits")
    Hv, dk = w.n_v_heads, w.d_k
    if w.bits == "iid48":
        coin = torch.randint(0, 2, (Hv, dk), generator=g)
        return torch.where(coin == 1, 8, 4).to(torch.uint8)
    if w.bits in ("half48", "mix248"):
        out = torch.empty((Hv, dk), dtype=torch.uint8)
        if w.bits == "half48":
            widths = [8] * (dk // 2) + [4] * (dk - dk // 2)
        else:
            widths = [8] * (dk // 4) + [4] * (dk // 4) + [2] * (dk - dk // 2)
        wt = torch.tensor(widths, dtype=torch.uint8)
        for h in range(Hv):
            perm = torch.randperm(dk, generator=g)
            out[h, perm] = wt
        return out
    raise ValueError(f"bit map {w.bits} is not a pure draw")


def active_slots(w: Workload) -> torch.Tensor:
    """Slot ids of the ``batch`` active requests (int32): the first ``batch``
    entries of a seeded permutation of the pool, or the identity when the pool
    has exactly ``batch`` slots."""
    if w.n_slots == w.batch:
        return torch.arange(w.batch, dtype=torch.int32)
    perm = torch.randperm(w.n_slots, generator=_gen("cpu", w, 0, 0, "slots"))
    return perm[: w.batch].to(torch.int32).contiguous()


def rotation_slots(w: Workload) -> list[torch.Tensor]:
    """Disjoint ``batch``-sized subsets covering the pool (same permutation as
    ``active_slots``; subset 0 is the active set).  Cycling through them keeps
    successive steps from being served out of the last-level cache."""
    perm = torch.randperm(w.n_slots, generator=_gen("cpu", w, 0, 0, "slots")).to(torch.int32)
    n = w.n_slots // w.batch
    return [perm[i * w.batch:(i + 1) * w.batch].contiguous() for i in range(n)]


def gqa_head(w: Workload, h_v: int) -> int:
    """q/k head read by value head h_v (grouped heads share q and k)."""
    return h_v // (w.n_v_heads // w.n_qk_heads)


def tile_count(w: Workload) -> int:
    return w.batch * w.n_v_heads * w.layers


def pool_elements(w: Workload) -> int:
    return w.n_slots * w.n_v_heads * w.d_k * w.d_v * w.layers

