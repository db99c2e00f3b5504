"""Throughput of the MRA-2 forward pass on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME] [--all] [--no-cpu]

One step = one mra_attention_forward call (pool, coarse logits, selection with
the coarse term, tile pass) over the whole workload, inputs resident in HBM.
Prints one JSON line with tokens/s, the roofline of the dominant kernel (the
tile pass, timed with HIP events on the stream it runs on) and the float64
oracle timed on the host as a reported CPU baseline. Beside the headline it
reports MRA-2-s, the head-wide budget and the gradient pass (forward with log
normalisers, then the backward given the forward's block means) on the same
inputs.

The CPU leg also compares the GPU's output with the oracle's on the heads it
computed (max row-normwise error, rows whose selection differs by a near-tie)
and reports the approximation error of MRA-2 against exact softmax attention,
||Z_MRA - Z||_F / ||Z||_F (the paper's accuracy measure, Sec. 5), on one head.
With --all the same numbers are given for every workload in "workloads".
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0      # MI355X dense bf16 matrix peak
PEAK_F32_TFLOPS = 157.3        # MI355X fp32 matrix / vector peak
PEAK_HBM_GBS = 8000.0          # MI355X HBM3E


def tile_flops(w) -> float:
    """Algorithmic flops of the tile pass: per selected 32x32 tile, 2*32*32*d
    for c Q_x K_y^T and 2*32*32*d for P V_y."""
    return 4.0 * w.B * w.H * w.nb * w.budget * 32 * 32 * w.d


def coarse_flops(w) -> float:
    """Coarse logits and the low-resolution term: 2*nb*nb*d each per head."""
    return 4.0 * w.B * w.H * w.nb * w.nb * w.d


def backward_flops(w) -> float:
    """Algorithmic flops of the gradient pass's tile products: per selected
    tile the five 32x32xd products S = c Q_x K_y^T, dP = G_x V_y^T,
    dV += A^T G, dQ += dP K, dK += dP^T Q (2*32*32*d each). The kernels run
    seven: S and dP are formed in both the dQ and the dK/dV pass."""
    return 10.0 * w.B * w.H * w.nb * w.budget * 32 * 32 * w.d


# MI355X unit counts and clock used for the tile pass's model floors
CUS, SIMDS_PER_CU, CLOCK_HZ = 256, 4, 2.4e9
L1_BYTES_PER_CLK_CU = 59.0     # measured ceiling of L2 -> CU loads (direct-to-LDS or VGPR)


def tile_floors(w) -> dict:
    """Lower bounds (µs) of the tile pass from unit counts and clock, one per
    resource: matrix cores (the MFMA roofline), the vector ALU (per selected
    tile and lane: 16 exponentials at quarter rate plus, for bfloat16, 16 FMA,
    8 conversions and 8 row-sum dot products at full rate; float32: 16 FMA and
    16 adds), and the per-CU vector-memory path (the tile's K and V bytes at
    the measured L2 -> CU ceiling). The measured pass exceeds the largest."""
    tiles = w.B * w.H * w.nb * w.budget
    e = 2 if w.dtype == "bf16" else 4
    peak = PEAK_BF16_TFLOPS if w.dtype == "bf16" else PEAK_F32_TFLOPS
    mfma = tile_flops(w) / (peak * 1e12) * 1e6
    valu_cycles = 16 * 16 + 32 * 4                          # per tile, one SIMD (wave64 on 16 lanes)
    valu = tiles * valu_cycles / (CUS * SIMDS_PER_CU * CLOCK_HZ) * 1e6
    vmem = tiles * 2 * 32 * w.d * e / (CUS * L1_BYTES_PER_CLK_CU * CLOCK_HZ) * 1e6
    return {"mfma_us": mfma, "valu_us": valu, "vector_memory_us": vmem}


def raw_tiles(w) -> bool:
    """The forward's tile pass reads K/V tiles from the rows themselves
    (bfloat16, float32 with d <= 64); for float32 with d = 128 pooling also
    writes a packed copy of K and V."""
    return w.dtype == "bf16" or w.d <= 64


def pool_bytes(w, packed=None) -> float:
    """Pooling pass: Q, K, V read once and the pooled rows written; in the
    forward for float32 (packed=None follows the forward) K and V are written
    once more in matrix-core operand order."""
    e = 2 if w.dtype == "bf16" else 4
    if packed is None:
        packed = not raw_tiles(w)
    copies = 5 if packed else 3
    return copies * w.B * w.H * w.n * w.d * e + 3 * w.B * w.H * w.nb * w.d * 4


TILE_SOURCES = ["paper_2207_10284_amd/csrc/tile.hip", "paper_2207_10284_amd/csrc/tile_ops.h",
                "paper_2207_10284_amd/csrc/common.h", "paper_2207_10284_amd/csrc/kernels.h"]
PROFILE = "profiles/tile_stream_kernel_base-4096.md"


def tile_source_hash() -> str:
    """Hash of the tile kernel's code: its sources with // comments and blank
    lines removed, so that editing a comment keeps recorded counters valid."""
    h = hashlib.sha256()
    for rel in TILE_SOURCES:
        with open(os.path.join(ROOT, rel)) as f:
            for line in f:
                code = line.split("//", 1)[0].rstrip()
                if code:
                    h.update(code.encode() + b"\n")
    return h.hexdigest()


def recorded_traffic():
    """HBM bytes per tile-kernel launch from the committed counter summary
    (FETCH_SIZE + WRITE_SIZE, calibrated), or None when the kernel source has
    changed since those counters were taken."""
    try:
        text = open(os.path.join(ROOT, PROFILE)).read()
    except OSError:
        return None
    h = re.search(r"tile_source_sha256:\s*([0-9a-f]{64})", text)
    t = re.search(r"tile_traffic_bytes_per_launch:\s*([0-9.eE+]+)", text)
    if not h or not t or h.group(1) != tile_source_hash():
        return None
    return float(t.group(1))


def time_launches(fn, iters: int, warmup: int = 3) -> float:
    """Average duration (ms) of `fn` (kernel launches on torch's current
    stream) between HIP events recorded on that stream."""
    import torch
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    s.record()
    for _ in range(iters):
        fn()
    e.record()
    torch.cuda.synchronize()
    return s.elapsed_time(e) / iters


def time_graph(fn, reps: int = 50, replays: int = 5) -> float:
    """Average duration (ms) of `fn` for kernels too short for Python to keep
    the GPU busy launch by launch: `reps` calls captured in one HIP graph,
    replayed, timed with HIP events on the capturing stream."""
    import torch
    fn()
    torch.cuda.synchronize()
    st = torch.cuda.Stream()
    st.wait_stream(torch.cuda.current_stream())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(st):
        with torch.cuda.graph(g, stream=st):
            for _ in range(reps):
                fn()
    torch.cuda.synchronize()
    g.replay()
    torch.cuda.synchronize()
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    cur = torch.cuda.current_stream()
    s.record(cur)
    for _ in range(replays):
        g.replay()
    e.record(cur)
    torch.cuda.synchronize()
    return s.elapsed_time(e) / (replays * reps)


def select_bytes(w) -> float:
    """The step-wise selection (mra_select): reads the coarse logits, writes
    the selected indices."""
    return 4.0 * w.B * w.H * w.nb * w.nb + 4.0 * w.B * w.H * w.nb * w.budget


def backward_leg(w, ops, tq, tk, tv, out, idx, ws, iters):
    """The gradient pass on the workload: mra_attention_backward alone (it
    pools q, k, v again), the backward given the forward's block means
    (mra_attention_backward_pooled), and a forward that also writes the log
    normalisers followed by that backward (one training step of the attention
    layer). Output gradient G ~ N(0, 1)."""
    import torch
    from paper_2207_10284_amd import inputs
    dev = tq.device
    lse = torch.empty(w.B, w.H, w.n, dtype=torch.float32, device=dev)
    g = np.random.Generator(np.random.PCG64(w.seed + 7)).standard_normal(tq.shape)
    g = inputs.round_to_bf16(g) if w.dtype == "bf16" else g.astype(np.float32)
    tg = torch.from_numpy(g).to(dev).to(tq.dtype)
    bws = torch.empty(ops.backward_workspace_bytes(w.B, w.H, w.n, w.d, tq.dtype), dtype=torch.uint8, device=dev)
    dq, dk, dv = (torch.empty_like(tq) for _ in range(3))

    def fwd():
        ops.attention_forward(tq, tk, tv, w.budget, out=out, idx_out=idx, workspace=ws, lse_out=lse)

    def bwd():
        ops.attention_backward(tq, tk, tv, out, tg, lse, idx, dq=dq, dk=dk, dv=dv, workspace=bws)

    pooled = ops.forward_pooled_rows(ws, w.B, w.H, w.n, w.d)      # views of the forward's workspace

    def bwd_pooled():
        ops.attention_backward(tq, tk, tv, out, tg, lse, idx, dq=dq, dk=dk, dv=dv, workspace=bws, pooled=pooled)

    fwd()
    bwd_ms = time_launches(bwd, iters)
    bwdp_ms = time_launches(bwd_pooled, iters)
    fb_ms = time_launches(lambda: (fwd(), bwd_pooled()), iters)
    tf = backward_flops(w) / (bwd_ms * 1e-3) / 1e12
    return {"ms_per_step": bwd_ms, "pooled_given_ms_per_step": bwdp_ms, "fwd_bwd_ms": fb_ms,
            "fwd_bwd_tokens_per_s": w.B * w.n / (fb_ms * 1e-3),
            "tile_tflops": tf, "tile_flops_per_step": backward_flops(w),
            "workspace_bytes": bws.numel()}


def cpu_baseline(w, q, k, v, gpu_out=None, gpu_idx=None, budget_s=25.0):
    """The float64 oracle (factored form, as it stands) over the heads of the
    workload, timed on the host until about `budget_s` seconds have passed.
    Returns (the cpu_baseline object, a parity object or None).

    Parity (outside the timed region): for every head the oracle computed,
    the GPU's selection against the oracle's (rows that differ, each
    difference a near-tie of the m-th score within 1e-6 relative) and the
    GPU's output against the oracle evaluated under the GPU's selection (max
    row-normwise relative error)."""
    from oracle import mra_oracle as O
    try:
        import threadpoolctl
        threads = max(i.get("num_threads", 1) for i in threadpoolctl.threadpool_info()) or 1
    except Exception:                                  # pragma: no cover
        threads = os.cpu_count() or 1
    t0 = time.perf_counter()
    done = []
    for b in range(w.B):
        for h in range(w.H):
            Z, I = O.mra_factored(q[b, h], k[b, h], v[b, h], 32, w.budget)
            done.append((b, h, Z, I))
            if time.perf_counter() - t0 > budget_s:
                break
        else:
            continue
        break
    dt = time.perf_counter() - t0
    heads = len(done)
    tokens = heads / w.H * w.n                         # tokens of a full H-head layer
    cpu = {"value": tokens / dt, "unit": "tokens/s", "cores": int(threads), "host_cpus": os.cpu_count(),
           "kind": "oracle",
           "sample": f"{heads} of {w.B * w.H} heads ({w.name}), float64 factored form, {dt:.1f} s"}
    if gpu_out is None:
        return cpu, None
    worst, tie_rows, rows = 0.0, 0, 0
    for b, h, Z, I in done:
        gi = gpu_idx[b, h]
        differ = [x for x in range(w.nb) if not np.array_equal(gi[x], I[x])]
        if differ:
            S = O.coarse_logits(O.block_mean(q[b, h], 32), O.block_mean(k[b, h], 32))
            for x in differ:
                tau = np.sort(S[x])[::-1][w.budget - 1]
                scale = max(abs(tau), np.abs(S[x]).max())
                for y in set(gi[x].tolist()) ^ set(I[x].tolist()):
                    if not abs(S[x, y] - tau) <= 1e-6 * scale:
                        raise AssertionError(f"{w.name}: selection of head ({b},{h}) row {x} differs beyond a tie")
            Z, _, _ = O.mra_factored_rows(q[b, h], k[b, h], v[b, h], 32, w.budget, idx=gi)
        tie_rows += len(differ)
        rows += w.nb
        got = gpu_out[b, h].astype(np.float64)
        num = np.abs(got - Z).max(axis=-1)
        den = np.maximum(np.abs(Z).max(axis=-1), 1e-30)
        worst = max(worst, float((num / den).max()))
    parity = {"max_row_rel_err": worst, "bar": 1e-5 if w.dtype == "f32" else 2e-2, "block_rows": rows,
              "heads": heads, "tie_swap_rows": tie_rows,
              "reference": "float64 oracle under the GPU's selection"}
    return cpu, parity


def approximation_error(w, q, k, v, gpu_out, b=0, h=0):
    """||Z_MRA - Z_exact||_F / ||Z_exact||_F of one head, Z_MRA the GPU's
    output and Z_exact softmax attention computed by the float64 oracle in
    slabs of rows (part of the CPU leg)."""
    from oracle import mra_oracle as O
    qh, kh, vh = (a[b, h].astype(np.float64) for a in (q, k, v))
    num = den = 0.0
    step = 1024
    for i0 in range(0, w.n, step):
        Ze = O.exact_attention_rows(qh, kh, vh, i0, min(i0 + step, w.n))
        dz = gpu_out[b, h, i0:i0 + step].astype(np.float64) - Ze
        num += float((dz ** 2).sum())
        den += float((Ze ** 2).sum())
    return {"value": float(np.sqrt(num / den)), "head": [b, h],
            "measure": "||Z_MRA-2 - softmax(QK^T/sqrt(d))V||_F / ||softmax(QK^T/sqrt(d))V||_F"}


def workload_line(w, ops, steps, warmup, cpu):
    """Forward, tile pass and pooling of one workload (its own inputs), and
    with `cpu` the CPU leg: oracle time, parity and approximation error."""
    import torch
    from paper_2207_10284_amd import inputs
    q, k, v = inputs.make_qkv(w)
    tdt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    dev = torch.device("cuda:0")
    tq, tk, tv = (torch.from_numpy(a).to(dev).to(tdt) for a in (q, k, v))
    out = torch.empty_like(tq)
    idx = torch.empty(w.B, w.H, w.nb, w.budget, dtype=torch.int32, device=dev)
    ws = torch.empty(ops.forward_workspace_bytes(w.B, w.H, w.n, w.d, w.budget, tdt), dtype=torch.uint8, device=dev)
    step = lambda: ops.attention_forward(tq, tk, tv, w.budget, out=out, idx_out=idx, workspace=ws)
    ms = time_launches(step, steps, warmup)
    qp, kp, vp = ops.pool(tq, tk, tv)
    S = ops.coarse_scores(qp, kp)
    sel = ops.select(S, w.budget)
    cm, cs, cv = ops.coarse_term(S, sel, vp)
    tile_out = torch.empty_like(tq)
    it = max(steps, 20)
    tile_ms = time_launches(lambda: ops.block_sddmm_spmm(tq, tk, tv, sel, cm, cs, cv, out=tile_out), it)
    pool_ms = time_launches(lambda: ops.pool(tq, tk, tv), it)
    peak = PEAK_BF16_TFLOPS if w.dtype == "bf16" else PEAK_F32_TFLOPS
    line = {"B": w.B, "H": w.H, "n": w.n, "d": w.d, "dtype": w.dtype, "budget": w.budget,
            "forward_us": ms * 1e3, "tokens_per_s": w.B * w.n / (ms * 1e-3),
            "tile_us": tile_ms * 1e3, "tile_frac_of_peak": tile_flops(w) / (tile_ms * 1e-3) / 1e12 / peak,
            "tile_peak_tflops": peak,
            "pool_frac_of_hbm": pool_bytes(w, packed=False) / (pool_ms * 1e-3) / 1e9 / PEAK_HBM_GBS}
    if cpu:
        torch.cuda.synchronize()
        out_h = out.float().cpu().numpy()
        gi = idx.cpu().numpy().astype(np.int64)
        c, par = cpu_baseline(w, q, k, v, out_h, gi, budget_s=10.0)
        line["cpu_baseline"] = c
        line["parity"] = par
        line["approximation_error"] = approximation_error(w, q, k, v, out_h, w.B - 1, w.H - 1)
    return line


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    # about 0.3 s of forward steps: the GPU reaches its sustained clock only
    # after some milliseconds of work (20 warm-up steps measure ~9% slower)
    ap.add_argument("--warmup", type=int, default=2000)
    ap.add_argument("--workload", default=None)
    ap.add_argument("--all", action="store_true",
                    help="also measure every other workload (forward, tile pass, pooling, CPU leg) into 'workloads'")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU-baseline leg")
    ap.add_argument("--no-variants", action="store_true",
                    help="skip timing MRA-2-s, the head-wide budget and the backward (profiling runs)")
    ap.add_argument("--backward-only", action="store_true",
                    help="time only the forward with log normalisers and the backward (profiling runs)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (the path has no multi-GPU mode); got --gpus {args.gpus}",
              file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2207_10284_amd import inputs, ops

    ops.load()
    w = inputs.WORKLOADS[args.workload or inputs.BENCH_WORKLOAD]
    q, k, v = inputs.make_qkv(w)
    tdt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    dev = torch.device("cuda:0")
    tq, tk, tv = (torch.from_numpy(a).to(dev).to(tdt) for a in (q, k, v))
    out = torch.empty_like(tq)
    idx = torch.empty(w.B, w.H, w.nb, w.budget, dtype=torch.int32, device=dev)
    ws = torch.empty(ops.forward_workspace_bytes(w.B, w.H, w.n, w.d, w.budget, tdt), dtype=torch.uint8, device=dev)
    torch.cuda.synchronize()

    def step():
        ops.attention_forward(tq, tk, tv, w.budget, out=out, idx_out=idx, workspace=ws)

    if args.backward_only:
        print(json.dumps({"backward": backward_leg(w, ops, tq, tk, tv, out, idx, ws, args.steps)}), flush=True)
        return

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    s.record()
    for _ in range(args.steps):
        step()
    e.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms = s.elapsed_time(e) / args.steps
    tokens_per_s = w.B * w.n / (ms * 1e-3)

    # The sparse-only variant MRA-2-s (Sec. 5) on the same inputs: reported
    # beside the headline, which is MRA-2.
    variants = {}
    if not args.no_variants:
        sparse_ms = time_launches(lambda: ops.sparse_attention_forward(tq, tk, tv, w.budget, out=out, idx_out=idx,
                                                                       workspace=ws), max(args.steps, 20))
        variants["mra2s"] = {"ms_per_step": sparse_ms, "tokens_per_s": w.B * w.n / (sparse_ms * 1e-3)}

    # MRA-2 with the head-wide budget of Alg. 1 (same total: m * nb blocks per
    # head, the nb diagonal blocks as priors), reported beside the headline.
    if not args.no_variants:
        gidx = torch.empty(w.B, w.H, w.nb, w.nb, dtype=torch.int32, device=dev)
        gws = torch.empty(ops.forward_global_workspace_bytes(w.B, w.H, w.n, w.d, tdt), dtype=torch.uint8, device=dev)
        gb = w.budget * w.nb - w.nb
        global_ms = time_launches(lambda: ops.attention_forward_global(tq, tk, tv, gb, True, out=out, idx_out=gidx,
                                                                       workspace=gws), max(args.steps, 20))
        variants["mra2_global_budget"] = {"ms_per_step": global_ms, "tokens_per_s": w.B * w.n / (global_ms * 1e-3),
                                          "budget_per_head": gb, "prior": "diagonal"}

    # Three resolutions R = {s0, 32, 1} (Alg. 1 with two refinement levels),
    # the second-level budget the headline's, reported beside it.
    if not args.no_variants:
        s0, m1 = inputs.MULTILEVEL[w.name]
        mws = torch.empty(ops.forward_multilevel_workspace_bytes(w.B, w.H, w.n, w.d, s0, m1, w.budget, tdt),
                          dtype=torch.uint8, device=dev)
        ml_ms = time_launches(lambda: ops.attention_forward_multilevel(tq, tk, tv, s0, m1, w.budget, out=out,
                                                                       idx2_out=idx, workspace=mws),
                              max(args.steps, 20))
        variants["mra_multilevel"] = {"ms_per_step": ml_ms, "tokens_per_s": w.B * w.n / (ml_ms * 1e-3),
                                      "coarse_block": s0, "budget1": m1, "budget2": w.budget}

    # Four resolutions R = {s_0, s_1, 32, 1} (Alg. 1 refined level by level).
    if not args.no_variants:
        scales, budgets = inputs.LEVELS[w.name]
        lws = torch.empty(ops.forward_levels_workspace_bytes(w.B, w.H, w.n, w.d, scales, budgets, tdt),
                          dtype=torch.uint8, device=dev)
        lv_ms = time_launches(lambda: ops.attention_forward_levels(tq, tk, tv, scales, budgets, out=out,
                                                                   workspace=lws), max(args.steps, 20))
        variants["mra_levels"] = {"ms_per_step": lv_ms, "tokens_per_s": w.B * w.n / (lv_ms * 1e-3),
                                  "scales": list(scales), "budgets": list(budgets)}

    if not args.no_variants:
        variants["backward"] = backward_leg(w, ops, tq, tk, tv, out, idx, ws, max(args.steps, 20))

    # Dominant kernel: the tile pass on the same inputs, timed alone: the
    # forward's own instantiation (raw K/V tiles) for every workload here.
    qp, kp, vp = ops.pool(tq, tk, tv)
    S = ops.coarse_scores(qp, kp)
    sel = ops.select(S, w.budget)
    cm, cs, cv = ops.coarse_term(S, sel, vp)
    tile_out = torch.empty_like(tq)
    it = max(args.steps, 20)
    tile_ms = time_launches(lambda: ops.block_sddmm_spmm(tq, tk, tv, sel, cm, cs, cv, out=tile_out), it)
    pool_ms = time_launches(lambda: ops.pool(tq, tk, tv), it)
    coarse_ms = time_launches(lambda: ops.coarse_scores(qp, kp), it)
    select_ms = time_graph(lambda: ops.select(S, w.budget))
    select_gbs = select_bytes(w) / (select_ms * 1e-3) / 1e9
    tflops = tile_flops(w) / (tile_ms * 1e-3) / 1e12
    peak = PEAK_BF16_TFLOPS if w.dtype == "bf16" else PEAK_F32_TFLOPS
    pool_gbs = pool_bytes(w, packed=False) / (pool_ms * 1e-3) / 1e9

    res = {
        "metric": "MRA-2 attention fwd tokens/s at n=4096,d=64 bf16; % MFMA peak on tile path",
        "value": tokens_per_s, "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": w.dtype, "data": "synthetic",
        "config": {"workload": w.name, "B": w.B, "H": w.H, "n": w.n, "d": w.d, "block": 32,
                   "budget": w.budget, "inputs": w.kind},
        "roofline": {"bound": "mfma", "kernel": "tile_stream_kernel (block-sparse SDDMM + SpMM + merge)",
                     "achieved": tflops, "peak": peak, "unit": "TFLOP/s", "frac": tflops / peak,
                     "traffic": recorded_traffic(), "traffic_unit": "bytes per launch",
                     "launch_us": tile_ms * 1e3,
                     "flops_per_launch": tile_flops(w)},
        # each stage launched alone, back to back (inputs warm in the caches);
        # in-step durations of the three forward kernels are in the profiles
        "stages_us": {"pool": pool_ms * 1e3, "tile": tile_ms * 1e3,
                      "coarse_scores_stepwise": coarse_ms * 1e3},
        "tile_floors": tile_floors(w),
        "pool_roofline": {"bound": "hbm", "achieved": pool_gbs, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                          "frac": pool_gbs / PEAK_HBM_GBS, "bytes_per_launch": pool_bytes(w, packed=False)},
        # the step-wise selection alone (the forward fuses it with the coarse
        # logits and the coarse term, so S~ never reaches HBM there). A
        # per-row radix search whose time is its latency, not its bytes: the
        # HBM fraction is reported for reference only.
        "select_roofline": {"bound": "latency", "kernel": "rows_kernel, select-only mode (mra_select)",
                            "achieved": select_gbs, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                            "frac": select_gbs / PEAK_HBM_GBS, "bytes_per_launch": select_bytes(w),
                            "launch_us": select_ms * 1e3,
                            "note": "latency-bound radix search; bytes at the HBM peak would take "
                                    f"{select_bytes(w) / (PEAK_HBM_GBS * 1e9) * 1e6:.2f} us"},
        **variants,
        "tflops_step": (tile_flops(w) + coarse_flops(w)) / (ms * 1e-3) / 1e12,
        "wall_s_timed": wall,
    }
    if not args.no_cpu:
        torch.cuda.synchronize()
        out_h = out.float().cpu().numpy()
        gi = idx.cpu().numpy().astype(np.int64)
        res["cpu_baseline"], res["parity"] = cpu_baseline(w, q, k, v, out_h, gi)
        res["approximation_error"] = approximation_error(w, q, k, v, out_h, w.B - 1, w.H - 1)
    if args.all:
        res["workloads"] = {}
        for name, ow in inputs.WORKLOADS.items():
            if name == w.name:
                continue
            print(f"# workload {name}", file=sys.stderr, flush=True)
            res["workloads"][name] = workload_line(ow, ops, max(args.steps, 20), 200, not args.no_cpu)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
