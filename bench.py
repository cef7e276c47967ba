"""Decode-step throughput of the quantized gated-Delta state pool on one MI355X.

Default workload (pool_b512): a 2048-slot pool, 512 active requests x 32
heads, d_k = d_v = 128, 6-bit mixed {4,8} codes with fp32 row/column scales,
bf16 activations.  One "step" is one fused decode launch over all 16,384
active (request, head) tiles.  By default successive steps rotate over four
disjoint 512-slot subsets of the pool (832 MiB cycle), so a step's 208 MiB
of state is not still resident in the 256 MB last-level cache from the
previous one; --resident keeps one subset (reported as cache-resident).

--workload pool_4bit: 512 active of a 2048-slot pool (rotated the same way),
32 heads, {2,4,8} codes at 4.0 bits per element, heavy-tailed states.
--workload stack48: 48 layers x 256 requests x 32 value heads (16 q/k heads),
6-bit {4,8}; one step is one replay of a HIP graph holding the 48 per-layer
launches (the 5.2 GB of packed state is far beyond the last-level cache).

Prints one JSON line (rank 0):
  value      state-updates/s (tiles advanced per second) over the timed steps
  roofline   the decode kernel's algorithmic state bytes per launch (codes
             read + codes written + scales read) / its mean launch duration
             (HIP events around the K back-to-back timed launches, gaps
             included), against the 8 TB/s HBM peak
  runs       the K timed steps split into --runs back-to-back runs (one
             event at each boundary): per-run ms per step, median, min, max
  bandwidth_refs  outside the timed region: a plain device copy of the
             launch's state bytes, and the library's memory-only reference
             of the decode launch (stepq_decode_stream_ref: same slots,
             workgroup order and traffic, no arithmetic), with the decode
             kernel's time over the reference's
  cpu_baseline  the fp64 oracle on the host cores on a bounded sample
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0
# fp32 vector peak, an FMA counted as one operation: 256 CUs x 4 SIMDs x 32
# lanes x 2.4 GHz = 78.6 Top/s (the published 157.3 TFLOP/s fp32 vector rate
# counts an FMA as two).  On gfx950 only plain fp32 add, subtract, multiply
# and FMA issue at that rate (a wave64 instruction every 2 cycles, without
# packed math); conversions, clamps (med3, max, min), round-to-integer,
# mixed-precision FMAs, byte packing, shifts and DPP moves issue at half of it
# (measured), and the decode steps are mostly made of those.
VALU_PEAK_TOPS = 256 * 4 * 32 * 2.4e9 / 1e12
# fp32 operations per state element of one step, counted from the method in
# its code-space form (each convert, add, multiply, FMA, max, round, clamp or
# pack counts one): decode 1, S^T k and S^T q 2, new value 2, requantize 4;
# the refit adds the row-magnitude sum 1, rescale 1, column max 1, fixed code
# 2 and the two least-squares sums 3.
# The row-absmax baseline adds the row maximum 1 and the rescale 1.
# The compiled bodies of every mode run S^T k and S^T q on the matrix cores
# (4x4x4 binary16 blocks), so those 2 operations are not VALU work there.
OPS_PER_ELEMENT = {False: 9, True: 17, "row_absmax": 11}
MATRIX_CORE_OPS = {False: 2, True: 2, "row_absmax": 2}
METRIC = "state-updates/s and achieved HBM GB/s (% of peak), B=512 heads=32 dk=dv=128"
CSRC = os.path.join(ROOT, "paper_2609_38169_amd", "csrc")


def mode_name(mode) -> str:
    return {False: "decode", True: "refit", "row_absmax": "rowmax"}[mode]


def traffic_file(mode, kda: bool, workload: str = "pool_b512", pivots: bool = False, calibrated=None) -> str:
    name = (mode_name(mode) + ("_kda" if kda else "") + ("_pivots" if pivots else "")
            + (f"_calibrated_{calibrated}" if calibrated else ""))
    return os.path.join(ROOT, "profiles", f"traffic_{name}_{workload}.json")


def kernel_sources(mode):
    files = ["stepq_device.h", "stepq_internal.h", "stepq_layout.h"]
    files += {False: ["stepq_kernels.hip"], True: ["stepq_refit_body.h", "stepq_refit.hip"],
              "row_absmax": ["stepq_refit_body.h", "stepq_rowmax.hip"]}[mode]
    return [os.path.join(CSRC, f) for f in files]


def log(msg: str):
    print(f"bench: {msg}", file=sys.stderr, flush=True)


def source_code(path: str) -> bytes:
    """A C++ source without its comments and blank lines (string literals
    in these sources hold no comment markers)."""
    import re
    text = open(path, encoding="utf-8").read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    text = re.sub(r"//[^\n]*", "", text)
    return "\n".join(line.rstrip() for line in text.splitlines() if line.strip()).encode()


def kernel_hash(mode=False) -> str:
    """Hash of the code of the timed kernel's sources (comments and blank
    lines left out), to tell whether committed counter summaries were taken
    on it."""
    h = hashlib.sha256()
    for f in kernel_sources(mode):
        h.update(source_code(f))
    return h.hexdigest()[:16]


def state_bytes_per_tile(bits_row, d_k, d_v, refit: bool = False) -> int:
    """Algorithmic bytes one tile update moves: its codes (and binary16
    pivot rows) read and written once, its fp32 row and column scales read
    once (and written once more when the step refits them).  A head held
    entirely in FP16 has no scales to read or fit."""
    import numpy as np
    n16 = int(np.sum(bits_row == 16))
    n8 = int(np.sum(bits_row == 8)); n4 = int(np.sum(bits_row == 4)); n2 = int(np.sum(bits_row == 2))
    code_bytes = (16 * n16 + 8 * n8 + 4 * n4 + 2 * n2) * d_v // 8
    if n16 == d_k:
        return 2 * code_bytes
    return 2 * code_bytes + (2 if refit else 1) * 4 * (d_k + d_v)


def cpu_baseline(w, bits, seconds: float):
    """The fp64 oracle on the host: decode steps on a sample of tiles of the
    same workload (layer 0) until ~seconds have elapsed."""
    import numpy as np
    import oracle
    from paper_2609_38169_amd import workloads as W
    rows = np.arange(16)                                  # 16 requests x 32 heads = 512 tiles
    slots = [int(s) for s in W.active_slots(w)[rows]]
    S = W.initial_state(w, 0, slots).numpy().reshape(-1, w.d_k, w.d_v)
    n = S.shape[0]
    tb = np.broadcast_to(bits[None], (len(rows),) + bits.shape).reshape(n, w.d_k)
    r, c = oracle.fit_absmax(S, bits=tb)
    # maps with FP16 pivot rows also carry the pivot values
    out = oracle.quantize(S.astype(np.float64), r, c, tb)
    codes, pv = out if isinstance(out, tuple) else (out, None)
    g = w.n_v_heads // w.n_qk_heads
    hq = np.arange(w.n_v_heads) // g
    # a few distinct steps of the sampled requests, drawn once and cycled
    steps_in = []
    for t in range(4):
        inp = W.step_inputs(w, 0, t)
        steps_in.append((inp["q"][rows].double().numpy()[:, hq].reshape(n, w.d_k),
                         inp["k"][rows].double().numpy()[:, hq].reshape(n, w.d_k),
                         inp["v"][rows].double().numpy().reshape(n, w.d_v),
                         inp["alpha"][rows].double().numpy().reshape(n),
                         inp["beta"][rows].double().numpy().reshape(n)))
    def timed(budget):
        nonlocal codes, pv
        done, step, elapsed = 0, 0, 0.0
        while elapsed < budget:
            q, k, v, a, b = steps_in[step % len(steps_in)]
            ts = time.perf_counter()
            res = oracle.decode_step(codes, r, c, tb, q, k, v, a, b, pv=pv)
            elapsed += time.perf_counter() - ts
            codes = res[0]
            if pv is not None:
                pv = res[-1]
            done += n
            step += 1
        return done / elapsed, step, elapsed

    cores = oracle.max_threads()
    value, step, elapsed = timed(seconds)
    oracle.set_threads(1)
    try:
        one, step1, elapsed1 = timed(seconds / 3)
    finally:
        oracle.set_threads(cores)
    return {"value": value, "unit": "state-updates/s", "cores": cores, "kind": "oracle",
            "sample": f"{step} decode steps x {n} tiles (16 requests x {w.n_v_heads} heads) of {w.name}, "
                      f"{elapsed:.1f} s of oracle time (4 distinct input steps cycled, draws excluded)",
            "single_core": {"value": one, "unit": "state-updates/s", "cores": 1,
                            "sample": f"{step1} decode steps of the same tiles, {elapsed1:.1f} s"}}


def traffic_entry(mode, kda: bool, workload: str = "pool_b512", pivots: bool = False, calibrated=None):
    """HBM bytes per launch (FETCH_SIZE + WRITE_SIZE, scaled by a plain
    copy's counters) from the committed rocprofv3 summary of this kernel,
    mode and workload, if it was taken on the current kernel source; else
    None."""
    try:
        t = json.load(open(traffic_file(mode, kda, workload, pivots, calibrated)))
    except (OSError, ValueError):
        return None
    if t.get("kernel_sha") != kernel_hash(mode):
        return None
    b = t.get("bytes_per_launch")
    return b.get("total") if isinstance(b, dict) else b


def adjacent_ids(ids) -> bool:
    """Whether a batch lists adjacent slots in increasing order (then the
    decode step gets the STEPQ_STEP_ADJACENT_SLOTS scheduling hint)."""
    d = ids[1:] - ids[:-1]
    return bool((d == 1).all().item()) if d.numel() else True


class Case:
    """One benchmark workload on the device: step(i) enqueues decode step i
    (launches_per_step kernel launches) on the current stream."""

    def __init__(self, **kw):
        self.__dict__.update(kw)


def pool_case(args, w, mode, dev):
    """A single-layer pool whose steps rotate over disjoint slot subsets."""
    import numpy as np
    import torch
    from paper_2609_38169_amd import workloads as W
    from paper_2609_38169_amd.pools import build_pool, row_bits

    bits = row_bits(w)
    row_weight = None
    if args.calibrated:
        # the calibration side of the setup step on this workload's own draws:
        # row units with 24 FP16 pivot rows (0.6% of the rows, as in the
        # paper's KDA setting) or head units with one whole FP16 head
        from paper_2609_38169_amd.calibrate import calibrate
        T = 8
        draws = [W.step_inputs(w, 0, 1000 + t) for t in range(T)]
        g = w.n_v_heads // w.n_qk_heads
        cat = lambda key: np.concatenate([d[key].float().numpy() for d in draws])
        cal = calibrate(np.repeat(cat("q"), g, axis=1), np.repeat(cat("k"), g, axis=1), cat("beta"), cat("alpha"),
                        W.initial_state(w, 0, range(4)).numpy(), budget=6.0, cand_bits=(4, 8), unit=args.calibrated,
                        n_pivots=24 if args.calibrated == "row" else 1, horizon=1024)
        bits, row_weight = cal.row_bits, cal.row_weight
    if args.pivots:
        # FP16 pivot rows: a seeded quarter of the heads keep 1-3 key rows in binary16
        bits = bits.copy()
        bits[W.pivot_mask_draw(w).numpy()] = 16
    if args.fp16_heads:
        # whole FP16 heads: a seeded choice of value heads keeps every row in binary16
        bits = bits.copy()
        bits[W.pivot_head_draw(w, 0, args.fp16_heads).numpy()] = 16
    log(f"building the {w.n_slots}-slot pool")
    pool = build_pool(w, device=dev, bits=bits, levels=args.levels)
    if row_weight is not None:
        pool.set_row_weight(row_weight)
    subsets = [s.to(dev) for s in (W.rotation_slots(w)[:1] if args.resident else W.rotation_slots(w))]
    if args.batch_order == "slot":
        # the same requests, listed in slot order: a request keeps its slot from step to step, so a
        # caller orders its batch once per change of composition; any order gives identical results
        subsets = [torch.sort(s).values for s in subsets]
    adjacent = [adjacent_ids(s) for s in subsets]
    n_inp = min(w.steps, args.steps + args.warmup)
    inputs = [W.step_inputs(w, 0, t, device=dev) for t in range(n_inp)]
    if args.kda:
        for t, inp in enumerate(inputs):
            inp["alpha"] = W.kda_gates(w, 0, t, device=dev)
    o = torch.empty((w.batch, w.n_v_heads, w.d_v), dtype=torch.float32, device=dev)
    prepared = {}      # one prepared call per (input step, slot subset) pair: arguments checked once

    def step(i):
        key = (i % n_inp, i % len(subsets))
        if key not in prepared:
            inp = inputs[key[0]]
            prepared[key] = pool.prepare_step(subsets[key[1]], inp["q"], inp["k"], inp["v"], inp["alpha"],
                                              inp["beta"], o, stream=torch.cuda.current_stream(), refit=mode,
                                              adjacent=adjacent[key[1]])
        prepared[key]()

    o_ref = torch.empty_like(o)
    prepared_ref = {}

    def ref(i):
        # the memory-only reference launch of step i (same slots, order and traffic; scalar gate read)
        j = i % len(subsets)
        if j not in prepared_ref:
            inp = W.step_inputs(w, 0, 0, device=dev)
            prepared_ref[j] = (inp, pool.prepare_stream_ref(subsets[j], inp["q"], inp["k"], inp["v"], inp["alpha"],
                                                            inp["beta"], o_ref, stream=torch.cuda.current_stream(),
                                                            adjacent=adjacent[j]))
        prepared_ref[j][1]()

    mix = {"pool_b512": "6-bit mixed {4,8}", "pool_4bit": "4-bit mixed {2,4,8}, heavy-tailed states"}[w.name]
    if args.calibrated:
        ints = bits[bits != 16]
        mix = (f"calibrated {args.calibrated} map ({ints.mean():.2f} bits/element on {(bits == 8).sum()} rows @8 and "
               f"{(bits == 4).sum()} @4, {(bits == 16).sum()} FP16 rows)")
    if args.pivots or args.fp16_heads:
        full = int((bits == 16).all(1).sum())
        rows = int((bits == 16).sum()) - full * w.d_k
        mix += f", {rows} FP16 pivot rows in {int(((bits == 16).any(1) & ~(bits == 16).all(1)).sum())} heads" if rows else ""
        mix += f", {full} of {w.n_v_heads} heads entirely FP16" if full else ""
    return Case(w=w, bits=bits, step=step, ref=ref, launches_per_step=1, n_subsets=len(subsets),
                keep=(pool, inputs, o, o_ref),
                tiles_per_step=w.batch * w.n_v_heads, layers=1,
                workload=f"{w.name}: {w.n_slots}-slot pool, B={w.batch} active, {w.n_v_heads} heads, "
                         f"d_k=d_v={w.d_k}, {mix}, fp32 scales, bf16 activations",
                extra={"slot_rotation": len(subsets), "cache_resident": bool(args.resident),
                       "batch_order": ("slot order (the drawn requests, listed by slot id)"
                                       if args.batch_order == "slot" else "as drawn"),
                       "adjacent_slots_hint": bool(all(adjacent))},
                pool_bytes=pool.pool_bytes)


def stack_case(args, w, mode, dev):
    """48 layer pools; one step is one graph replay of the 48 launches."""
    import numpy as np
    import torch
    from paper_2609_38169_amd import workloads as W
    from paper_2609_38169_amd.pools import build_pool, row_bits

    slots = W.active_slots(w).to(dev)
    pools, bufs, bits0 = [], [], None
    for L in range(w.layers):
        b = row_bits(w, L)
        bits0 = b if bits0 is None else bits0
        pools.append(build_pool(w, L, device=dev, bits=b, levels=args.levels))
        inp = W.step_inputs(w, L, 0, device=dev)
        if args.kda:
            inp["alpha"] = W.kda_gates(w, L, 0, device=dev)
        inp["o"] = torch.empty((w.batch, w.n_v_heads, w.d_v), dtype=torch.float32, device=dev)
        bufs.append(inp)
        if L % 8 == 7:
            log(f"{L + 1} of {w.layers} layer pools built")
    main_stream = torch.cuda.current_stream()
    side = torch.cuda.Stream()
    side.wait_stream(main_stream)
    graph = torch.cuda.CUDAGraph()
    adjacent = adjacent_ids(slots)
    with torch.cuda.stream(side):
        calls = [pools[L].prepare_step(slots, bufs[L]["q"], bufs[L]["k"], bufs[L]["v"], bufs[L]["alpha"],
                                       bufs[L]["beta"], bufs[L]["o"], stream=side, refit=mode, adjacent=adjacent)
                 for L in range(w.layers)]
        with torch.cuda.graph(graph, stream=side):
            for c in calls:
                c()
    main_stream.wait_stream(side)
    torch.cuda.synchronize()

    def step(i):
        graph.replay()

    o_ref = torch.empty_like(bufs[0]["o"])
    ref_call = []

    def ref(i):
        # the memory-only reference of one layer's launch (layer 0: same slots, order and traffic)
        if not ref_call:
            b = bufs[0]
            alpha = b["alpha"] if b["alpha"].dim() == 2 else b["alpha"][:, :, 0].contiguous()
            ref_call.append((alpha, pools[0].prepare_stream_ref(slots, b["q"], b["k"], b["v"], alpha, b["beta"], o_ref,
                                                                stream=torch.cuda.current_stream(), adjacent=adjacent)))
        ref_call[0][1]()

    pool_bytes = sum(p.pool_bytes for p in pools)
    fp32_bytes = w.layers * w.n_slots * w.n_v_heads * w.d_k * w.d_v * 4
    return Case(w=w, bits=bits0, step=step, ref=ref, launches_per_step=w.layers, n_subsets=1,
                keep=(pools, bufs, graph, calls, side, o_ref, ref_call), tiles_per_step=w.layers * w.batch * w.n_v_heads,
                layers=w.layers,
                workload=f"{w.name}: {w.layers} layers x B={w.batch} requests x {w.n_v_heads} value heads "
                         f"({w.n_qk_heads} q/k heads), d_k=d_v={w.d_k}, 6-bit mixed {{4,8}}, fp32 scales, "
                         f"bf16 activations, one HIP graph of {w.layers} launches per step",
                extra={"graph_launches_per_step": w.layers, "pool_bytes": pool_bytes, "fp32_pool_bytes": fp32_bytes,
                       "pool_compression": fp32_bytes / pool_bytes, "adjacent_slots_hint": adjacent},
                pool_bytes=pool_bytes)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=256)
    ap.add_argument("--warmup", type=int, default=16)
    ap.add_argument("--settle-ms", type=float, default=150.0,
                    help="untimed steps before the warmup until this much GPU time has elapsed (clock ramp)")
    ap.add_argument("--workload", choices=["pool_b512", "pool_4bit", "stack48"], default="pool_b512")
    ap.add_argument("--resident", action="store_true", help="no slot rotation (cache-resident number)")
    ap.add_argument("--calibrated", choices=["row", "head"], default=None,
                    help="pool workloads: the precision map from the calibration side of the setup step "
                         "(row units with 24 FP16 pivot rows, or head units with one FP16 head)")
    ap.add_argument("--batch-order", choices=["slot", "drawn"], default="slot",
                    help="pool workloads: list each step's active requests in slot order (default; a caller-side "
                         "choice, made once per batch composition: any order gives the same results), or in the "
                         "order they were drawn")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--runs", type=int, default=3,
                    help="the K timed steps are split into this many back-to-back runs; their median, min and max "
                         "per-step times are reported beside the whole-region figures")
    ap.add_argument("--no-copy-ref", action="store_true",
                    help="skip the bandwidth references (a plain device copy of the step's state bytes, and the "
                         "library's memory-only reference of the decode launch with the same slots and order)")
    ap.add_argument("--kda", action="store_true", help="channel-wise (KDA) gates [B][Hv][d_k] instead of alpha")
    ap.add_argument("--refit", action="store_true", help="online dual-axis refit of the scales in every step")
    ap.add_argument("--row-absmax", action="store_true",
                    help="requantize as the row-wise absmax INT-b baseline (row factors refit, column factors 1)")
    ap.add_argument("--pivots", action="store_true",
                    help="a seeded quarter of the heads keep 1-3 FP16 pivot rows (pool workloads)")
    ap.add_argument("--levels", type=int, choices=[0, 1], default=0,
                    help="level normalisation of the codes: 0 = N1 (q / q_b), 1 = N2 (2^(8-b) q, the KDA codebook)")
    ap.add_argument("--fp16-heads", type=int, default=0,
                    help="this many seeded value heads are kept entirely in FP16 (pool workloads)")
    args = ap.parse_args()

    if args.refit and args.row_absmax:
        print("--refit and --row-absmax exclude each other", file=sys.stderr)
        sys.exit(2)
    if (args.pivots or args.fp16_heads or args.calibrated) and args.workload == "stack48":
        print("--pivots, --fp16-heads and --calibrated apply to the single-layer pool workloads", file=sys.stderr)
        sys.exit(2)
    mode = True if args.refit else ("row_absmax" if args.row_absmax else False)
    rescale = bool(mode)          # the step writes the scales back
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the library has no multi-GPU path (each (request, head) tile is "
              "independent, so heads or requests shard across GPUs with no exchange). Run with --gpus 1.",
              file=sys.stderr)
        sys.exit(2)

    import dataclasses
    import numpy as np
    import torch
    from paper_2609_38169_amd import workloads as W

    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    t_setup = time.perf_counter()
    if args.workload == "pool_b512":
        case = pool_case(args, W.workload(2), mode, dev)
    elif args.workload == "pool_4bit":
        # the 512-request workload on a 2048-slot pool, so that rotating slot
        # subsets keeps each step's state out of the last-level cache
        case = pool_case(args, dataclasses.replace(W.workload(3), n_slots=2048), mode, dev)
    else:
        case = stack_case(args, W.workload(4), mode, dev)
    w = case.w
    torch.cuda.synchronize()
    setup_s = time.perf_counter() - t_setup
    stream = torch.cuda.current_stream()
    LPS = case.launches_per_step

    log(f"setup done in {setup_s:.1f} s; settling clocks")
    # Settle: the GPU's clocks ramp up over the first ~50 ms of sustained
    # load (a step measured on a cold GPU is ~20% slower), so steps run
    # untimed until args.settle_ms of GPU time has elapsed; then the W
    # warmup steps; then the K timed steps.
    settle_n, settle_ms = 0, 0.0
    s0 = torch.cuda.Event(enable_timing=True)
    s1 = torch.cuda.Event(enable_timing=True)
    chunk = max(1, 64 // LPS)
    while settle_ms < args.settle_ms:
        s0.record(stream)
        for i in range(chunk):
            case.step(settle_n + i)
        s1.record(stream)
        torch.cuda.synchronize()
        settle_n += chunk
        settle_ms += s0.elapsed_time(s1)
    log(f"settled after {settle_n} untimed steps ({settle_ms:.0f} ms); warmup and timing")
    for i in range(args.warmup):
        case.step(i)
    torch.cuda.synchronize()

    K = args.steps
    for i in range(args.warmup, args.warmup + K):
        case.step(i)                    # prepare every call outside the timed region
    torch.cuda.synchronize()
    # timed region: K back-to-back steps between two events on the launch stream
    # (split into R back-to-back runs with an event at each boundary: the
    # per-run times give the run-to-run spread; the region is still exactly
    # K steps between its first and last event)
    R = max(1, min(args.runs, K))
    bounds = [K * j // R for j in range(R + 1)]
    tev = [torch.cuda.Event(enable_timing=True) for _ in range(R + 1)]
    tev[0].record(stream)
    for j in range(R):
        for i in range(bounds[j], bounds[j + 1]):
            case.step(args.warmup + i)
        tev[j + 1].record(stream)
    torch.cuda.synchronize()
    total_ms = tev[0].elapsed_time(tev[R])
    kern_ms = total_ms / (K * LPS)  # mean launch duration, gaps between launches included
    run_ms = [tev[j].elapsed_time(tev[j + 1]) / (bounds[j + 1] - bounds[j]) for j in range(R)]

    # diagnostics outside the timed region: one event pair per step
    n_diag = min(K, 64)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2 * n_diag)]
    for i in range(n_diag):
        ev[2 * i].record(stream)
        case.step(args.warmup + K + i)
        ev[2 * i + 1].record(stream)
    torch.cuda.synchronize()
    per_launch_ms = [ev[2 * i].elapsed_time(ev[2 * i + 1]) / LPS for i in range(n_diag)]
    nsub = case.n_subsets
    per_subset = [float(np.mean([per_launch_ms[i] for i in range(n_diag) if (args.warmup + K + i) % nsub == j] or [0.0]))
                  for j in range(nsub)]

    bits = case.bits
    per_tile = [state_bytes_per_tile(bits[h], w.d_k, w.d_v, rescale) for h in range(w.n_v_heads)]
    launch_bytes = w.batch * sum(per_tile)           # one launch = one layer of the step
    gate_elems = w.n_v_heads * (w.d_k if args.kda else 1)
    act_bytes = w.batch * (2 * w.n_qk_heads * w.d_k * 2 + w.n_v_heads * w.d_v * 2 + (gate_elems + w.n_v_heads) * 2
                           + w.n_v_heads * w.d_v * 4 + 4)
    achieved = launch_bytes / (kern_ms * 1e-3) / 1e9
    valu_ops = OPS_PER_ELEMENT[mode] - MATRIX_CORE_OPS[mode]
    valu_tops = w.batch * w.n_v_heads * w.d_k * w.d_v * valu_ops / (kern_ms * 1e-3) / 1e12
    value = case.tiles_per_step * K / (total_ms * 1e-3)
    state_gbps = launch_bytes * LPS * K / (total_ms * 1e-3) / 1e9
    kern_name = ("refit_kernel" if rescale else "decode_kernel") + ("<128, bf16, kda" if args.kda else "<128, bf16")
    kern_name += {True: ", dual axis", "row_absmax": ", row absmax", False: ""}[mode]
    kern_name += (", heads with pivots on the generic body" if args.pivots else "")
    kern_name += (", FP16 heads" if args.fp16_heads else "") + ">"

    line = {
        "metric": METRIC,
        "value": value,
        "unit": "state-updates/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": total_ms / K,
        "runs": {"n": R, "steps_each": [bounds[j + 1] - bounds[j] for j in range(R)], "ms_per_step": run_ms,
                 "median": float(np.median(run_ms)), "min": float(np.min(run_ms)), "max": float(np.max(run_ms))},
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32 (S^T k, S^T q: binary16 hi+lo matrix-core operands, fp32 accumulation)",
        "data": "synthetic",
        "config": dict({"workload": case.workload,
                        "gate": "channel-wise d [B][Hv][d_k] (KDA)" if args.kda else "scalar alpha [B][Hv] (GDN)",
                        "scales": {True: "online dual-axis refit every step", "row_absmax": "row-wise absmax every "
                                   "step (INT-b baseline)", False: "frozen"}[mode],
                        "levels": "N2: z = 2^(8-b) q" if args.levels else "N1: z = q / q_b"}, **case.extra),
        "GBps_state": state_gbps,
        "pct_hbm_peak": 100.0 * state_gbps / HBM_PEAK_GBPS,
        "roofline": {
            "bound": "hbm",
            "achieved": achieved,
            "peak": HBM_PEAK_GBPS,
            "unit": "GB/s",
            "frac": achieved / HBM_PEAK_GBPS,
            "traffic": traffic_entry(mode, args.kda, w.name, args.pivots, args.calibrated)
                       if not args.fp16_heads else None,
            "valu": {"achieved": valu_tops, "peak": VALU_PEAK_TOPS, "unit": "Top/s", "frac": valu_tops / VALU_PEAK_TOPS,
                     "ops_per_element": valu_ops, "matrix_core_ops_per_element": MATRIX_CORE_OPS[mode]},
            "kernel": kern_name,
            "kernel_ms_mean": kern_ms,
            "launches_per_step": LPS,
            "launch_ms_event_pairs": {"mean": float(np.mean(per_launch_ms)), "min": float(np.min(per_launch_ms)),
                                      "max": float(np.max(per_launch_ms)), "per_slot_subset": per_subset},
            "bytes_per_launch": launch_bytes,
            "activation_bytes_per_launch": act_bytes,
            "kernel_sha": kernel_hash(mode),
        },
        "setup_s": setup_s,
        "settle": {"steps": settle_n, "gpu_ms": settle_ms,
                   "why": "untimed steps before warmup until the GPU clocks reach steady state under load"},
    }
    if rescale or w.name == "pool_4bit":
        # Bound by VALU issue, not by HBM, so that roofline is the primary one: the refitting
        # steps, and the {2,4,8} pool, whose 2-bit rows carry four codes per byte (the library's
        # memory-only reference of the pool_4bit launch takes ~54 us against ~64 us for the full
        # kernel, and a copy of the kernel without the code-word traffic takes as long as the full
        # one; on pool_b512 and stack48 the memory-only reference is within a few percent).
        rl = line["roofline"]
        hbm = {k: rl[k] for k in ("achieved", "peak", "unit", "frac")}
        valu = rl.pop("valu")
        rl.update({"bound": "alu", "achieved": valu["achieved"], "peak": valu["peak"], "unit": valu["unit"],
                   "frac": valu["frac"], "ops_per_element": valu["ops_per_element"],
                   "matrix_core_ops_per_element": valu["matrix_core_ops_per_element"], "hbm": hbm})
    if not args.no_copy_ref:
        # achievable-bandwidth references, outside the timed region
        src = torch.empty(launch_bytes // 2, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        c0, c1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        c0.record(stream)
        for _ in range(20):
            dst.copy_(src)
        c1.record(stream)
        torch.cuda.synchronize()
        del src, dst
        refs = {"device_copy_GBps": 2 * (launch_bytes // 2) * 20 / (c0.elapsed_time(c1) * 1e-3) / 1e9,
                "device_copy": "torch copy of half the launch's state bytes (read + write = the launch's bytes)"}
        n_ref = 64
        for i in range(8):
            case.ref(i)
        c0.record(stream)
        for i in range(n_ref):
            case.ref(i)
        c1.record(stream)
        torch.cuda.synchronize()
        ref_ms = c0.elapsed_time(c1) / n_ref
        # the frozen step's bytes (codes read and written, scales read): the reference writes no scales
        ref_bytes = w.batch * sum(state_bytes_per_tile(bits[h], w.d_k, w.d_v, False) for h in range(w.n_v_heads))
        refs.update({"memory_only_us": ref_ms * 1e3, "memory_only_GBps": ref_bytes / (ref_ms * 1e-3) / 1e9,
                     "memory_only": "stepq_decode_stream_ref: the frozen decode launch's tiles, workgroup order and "
                                    "memory traffic (codes read and written back, scales and activations read, o "
                                    "written) without arithmetic, over the same slot subsets",
                     "kernel_over_memory_only": kern_ms / ref_ms})
        line["bandwidth_refs"] = refs
    if not args.no_cpu_baseline:
        log(f"GPU timing done ({total_ms / K * 1e3:.1f} us per step); oracle baseline on the host")
        line["cpu_baseline"] = cpu_baseline(w, bits, args.cpu_seconds)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
