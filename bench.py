"""Throughput of Reformer LSH attention on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]
                    [--cpu-budget S] [--copy-probe BYTES] [--sweep-length]

One step is one full forward pass over one batch of the workload: hash, sort,
chunked attention (with the gather fused into its staging) and the round
combine, each through the C ABI of liblsh on torch's current stream.  Inputs
are generated once and are resident in HBM before timing starts.  Prints one
JSON line with the whole-job tokens/s, the per-stage times (HIP events on the
stream the kernels run on), the roofline position of the dominant kernel and
the CPU oracle's rate on a bounded sample of the same workload.

The default workload is B=1, H=16, L=65536, d=64 (d_model 1024), bf16,
n_buckets=1024, 8 hashing rounds, chunks of 64, causal, with queries from a
mixture of 256 Gaussians.

Roofline.  The dominant stage (largest time) is placed against the MI355X
peak that bounds it: algorithmic work of the stage / the stage's average
duration (HIP events around the stage's one library call on the stream it
runs on).  `traffic` is the HBM traffic of that stage's kernels per call,
from rocprofv3 FETCH_SIZE and WRITE_SIZE counters recorded under profiles/
(scaled by what the same counters read for a plain device copy of known
size, which --copy-probe launches after the timed steps); it is null when
the kernel sources differ from the ones the counters were taken on.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np
import torch

from paper_2001_04451_amd import lsh
from paper_2001_04451_amd import workloads as W

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, GB/s
BF16_MFMA_PEAK_TFLOPS = 2500.0  # MI355X dense bf16 matrix peak, TFLOP/s
ROOT = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(ROOT, "paper_2001_04451_amd", "csrc")

# Stages as the library runs them: the kernels of each call, the source files
# they are built from, and the peak that bounds the stage's main kernel.
STAGES = {
    "hash": {"kernels": ["prep_r_cols_kernel", "prep_r_max_kernel", "hash_kernel",
                         "hash_refine_kernel"],
             "sources": ["hash.hip", "common.h"], "bound": "mfma", "work": "hash_flop"},
    "sort": {"kernels": ["sort_hist_kernel", "sort_scan_kernel", "sort_scatter_kernel"],
             "sources": ["sort.hip", "common.h"], "bound": "hbm", "work": "sort_bytes"},
    "attn": {"kernels": ["attn_prep_kernel", "attn_fwd_bf16_kernel"],
             "sources": ["attn_fwd.hip", "attn_common.h", "common.h"], "bound": "hbm",
             "work": "attn_bytes"},
    "bwd": {"kernels": ["bwd_prep_kernel", "bwd_strip_kernel", "bwd_reduce_kernel"],
            "sources": ["attn_bwd.hip", "attn_common.h", "common.h"], "bound": "hbm",
            "work": "bwd_bytes"},
    "combine": {"kernels": ["combine_kernel"], "sources": ["combine.hip", "common.h"],
                "bound": "hbm", "work": "combine_bytes"},
}


def sources_digest(files) -> str:
    h = hashlib.sha256()
    for f in files:
        with open(os.path.join(CSRC, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def recorded_traffic(workload: str, stage: str):
    """HBM bytes per call of the stage from the committed counter summary, or
    None when there is none or the stage's kernel sources have changed."""
    path = os.path.join(ROOT, "profiles", f"traffic_{workload}.json")
    if not os.path.exists(path):
        return None
    with open(path) as fh:
        rec = json.load(fh)
    st = rec.get("stages", {}).get(stage)
    if not st or st.get("sources") != sources_digest(STAGES[stage]["sources"]):
        return None
    return st["bytes_per_call"]


def algorithmic_work(w: W.Workload) -> dict:
    """Algorithmic work of each stage for one forward pass (not what the kernels
    actually move): flops of the contractions and bytes a minimal data flow
    must read and write."""
    rr = w.row_rounds
    e = 2 if w.dtype == "bf16" else 4
    d, m, n_r = w.d, w.chunk, w.n_rounds
    rows = w.rows
    return {
        # 2 * d * (n_b/2) flops per row-round for [xR; -xR]
        "hash_flop": rr * d * w.n_buckets,
        # QK^T and PV over a 2m-key window: 2 * (2m * d) * 2 flops per row-round
        "attn_flop": rr * 8 * m * d,
        # per row-round: q and v rows gathered, o_rounds row (fp16 for bf16
        # calls, with its exponent byte; fp32 for fp32 calls) and lse written,
        # the slot's position read, the token's bucket ids (two per 32-bit
        # word) gathered
        "attn_bytes": rr * (2 * d * e + e * d + (1 if e == 2 else 0) + 4 + 4
                            + 4 * ((n_r + 1) // 2)),
        # ids read twice, perm and undo written
        "sort_bytes": rr * 16,
        # per row: n_r o_rounds rows (+ exponent byte for bf16 calls), lse and
        # undo read, one output row and its log-partition written
        "combine_bytes": rows * (n_r * (e * d + 8 + (1 if e == 2 else 0)) + d * e + 4),
        # backward, recomputing the logits: S = QK^T, dP = dO V^T, dV += P^T dO,
        # dQ += dA K, dK += dA^T Q over the 2m-key window, 2 * (2m * d) flops each
        "bwd_flop": rr * 20 * m * d,
        # per row-round: q, v and dO rows gathered, the slot's position, the
        # token's total log-partition and D_i = dO_i . o_i; per row: out and
        # dout read once for D_i, dq and dv written in fp32
        "bwd_bytes": rr * (3 * d * e + 4 + 8) + rows * (2 * d * e + 2 * 4 * d),
    }


def run_gpu(w: W.Workload, steps: int, warmup: int, x: dict | None = None) -> dict:
    dev = torch.device("cuda:0")
    if x is None:
        x = W.make_inputs(w)
    tdt = torch.bfloat16 if w.dtype == "bf16" else torch.float32

    def up(a, bf):
        t = torch.from_numpy(np.ascontiguousarray(a))
        return (t.view(torch.int16).view(torch.bfloat16) if bf else t).to(dev)

    bf = w.dtype == "bf16"
    q, v, R = up(x["q"], bf), up(x["v"], bf), up(x["R"], False)
    dout = up(x["dout"], bf) if w.backward else None
    cfg = lsh.Config.of(w)
    B, H, L, nr, nb, d = w.B, w.H, w.L, w.n_rounds, w.n_buckets, w.d
    buckets = torch.empty((B, H, L, nr), dtype=torch.int32, device=dev)
    perm = torch.empty((B, H, nr, L), dtype=torch.int32, device=dev)
    undo = torch.empty_like(perm)
    bstart = torch.empty((B, H, nr, nb + 1), dtype=torch.int32, device=dev)
    o_r = torch.empty((B, H, nr, L, d), dtype=lsh.rounds_dtype(tdt), device=dev)
    o_e = torch.empty((B, H, nr, L), dtype=torch.uint8, device=dev) if bf else None
    lse_r = torch.empty((B, H, nr, L), dtype=torch.float32, device=dev)
    out = torch.empty((B, H, L, d), dtype=tdt, device=dev)
    lse = torch.empty((B, H, L), dtype=torch.float32, device=dev)
    ws_hash = torch.empty(max(256, lsh.workspace_bytes(cfg, tdt, lsh.LSH_OP_HASH)),
                          dtype=torch.uint8, device=dev)
    ws_sort = torch.empty(max(256, lsh.workspace_bytes(cfg, tdt, lsh.LSH_OP_SORT)),
                          dtype=torch.uint8, device=dev)
    ws_attn = torch.empty(max(256, lsh.workspace_bytes(cfg, tdt, lsh.LSH_OP_ATTN_FWD)),
                          dtype=torch.uint8, device=dev)

    stages = ["hash", "sort", "attn", "combine"]

    def step(ev=None):
        if ev is not None:
            ev[0].record()
        lsh.lsh_hash(cfg, q, R, buckets, ws_hash)
        if ev is not None:
            ev[1].record()
        lsh.lsh_sort_permute(cfg, buckets, ws_sort, perm, undo, bstart)
        if ev is not None:
            ev[2].record()
        lsh.lsh_chunk_attn_fwd(cfg, q, v, buckets, perm, bstart, o_r, o_e, lse_r, ws_attn)
        if ev is not None:
            ev[3].record()
        lsh.lsh_combine_rounds(cfg, o_r, o_e, lse_r, undo, tdt, out, lse)
        if ev is not None:
            ev[4].record()

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    events = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(steps):
        step(events[k])
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    per_stage = {s: float(np.mean([events[k][i].elapsed_time(events[k][i + 1])
                                   for k in range(steps)])) for i, s in enumerate(stages)}
    if not torch.isfinite(out.float()).all():
        raise RuntimeError("non-finite output")
    res = {"ms_per_step": (t1 - t0) * 1e3 / steps, "stage_ms": per_stage,
           "state": {"buckets": buckets, "perm": perm, "out": out}}
    if w.backward:
        # the backward on the last forward's state: one lsh_chunk_attn_bwd call
        # per step, timed the same way
        dq = torch.empty((B, H, L, d), dtype=torch.float32, device=dev)
        dv = torch.empty_like(dq)
        ws_bwd = torch.empty(max(256, lsh.workspace_bytes(cfg, tdt, lsh.LSH_OP_ATTN_BWD)),
                             dtype=torch.uint8, device=dev)

        def bwd():
            lsh.lsh_chunk_attn_bwd(cfg, q, v, out, dout, lse, buckets, perm, undo, bstart, dq, dv,
                                   ws_bwd)

        for _ in range(warmup):
            bwd()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        tb0 = time.perf_counter()
        e0.record()
        for _ in range(steps):
            bwd()
        e1.record()
        torch.cuda.synchronize()
        tb1 = time.perf_counter()
        if not (torch.isfinite(dq).all() and torch.isfinite(dv).all()):
            raise RuntimeError("non-finite gradients")
        res["bwd_ms"] = e0.elapsed_time(e1) / steps
        res["bwd_wall_ms"] = (tb1 - tb0) * 1e3 / steps
    return res


def cpu_model() -> str:
    """The host CPU's model name (as lscpu reports it)."""
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(w: W.Workload, budget_s: float, x: dict, state: dict) -> tuple[dict, dict]:
    """The oracle on whole (batch, head) slices of the benchmark batch, in a
    seeded random order, until the time budget is spent; rate scaled to the
    full workload's tokens.  The same slices of the GPU's last forward are
    compared with the oracle's: bucket ids bit for bit (near-tie row-rounds
    counted), the permutation, and the output's max-abs error."""
    import oracle  # test infrastructure: used here only for the reported baseline and check

    oracle.build()
    R = x["R"].astype(np.float64)
    total_slices = w.B * w.H
    order = np.random.default_rng(0).permutation(total_slices)
    gpu_b = state["buckets"].cpu().numpy()
    gpu_p = state["perm"].cpu().numpy()
    gpu_o = state["out"].float().cpu().numpy()
    slices, elapsed = 0, 0.0
    n_tie = n_mism = n_mism_outside = 0
    perm_equal, err = True, 0.0
    while slices < total_slices and (slices == 0 or elapsed < budget_s):
        b, h = divmod(int(order[slices]), w.H)
        q64 = W.as_f64(x["q"][b:b + 1, h:h + 1], w.dtype)
        v64 = W.as_f64(x["v"][b:b + 1, h:h + 1], w.dtype)
        t0 = time.perf_counter()
        ref = oracle.lsh_attention_fwd(q64, v64, R, w.chunk, w.causal)
        elapsed += time.perf_counter() - t0
        slices += 1
        mism = gpu_b[b:b + 1, h:h + 1] != ref["buckets"]
        n_tie += int(ref["near_tie"].sum())
        n_mism += int(mism.sum())
        n_mism_outside += int((mism & ~ref["near_tie"]).sum())
        perm_equal &= bool(np.array_equal(gpu_p[b:b + 1, h:h + 1], ref["perm"]))
        err = max(err, float(np.abs(gpu_o[b:b + 1, h:h + 1] - ref["out"]).max()))
    tokens = w.B * w.L * slices / total_slices
    base = {"value": tokens / elapsed, "unit": "tokens/s", "cores": oracle.num_threads(),
            "kind": "oracle", "cpu_model": cpu_model(),
            "sample": f"{slices} of {total_slices} (batch, head) slices of the benchmark batch "
                      f"(L={w.L}, n_rounds={w.n_rounds}), fp64, {elapsed:.1f} s of oracle time; "
                      f"tokens/s scaled by the slice fraction"}
    parity = {"slices": slices, "near_tie_row_rounds": n_tie, "bucket_mismatches": n_mism,
              "bucket_mismatches_outside_near_ties": n_mism_outside, "perm_equal": perm_equal,
              "out_max_abs_err": err, "tol": 2e-2 if w.dtype == "bf16" else 1e-5}
    return base, parity


def stage_rooflines(w: W.Workload, work: dict, st: dict) -> dict:
    """Each forward stage against the roof that bounds it, from its algorithmic
    work and its measured time: the hash and the chunk attention on the bf16
    matrix peak (the attention also on HBM, its bound by arithmetic
    intensity), the sort and the combine (the scatter back) on HBM."""
    def mfma(flop, ms):
        a = flop / (ms * 1e-3) / 1e12
        return {"bound": "mfma", "achieved": a, "peak": BF16_MFMA_PEAK_TFLOPS,
                "unit": "TFLOP/s", "frac": a / BF16_MFMA_PEAK_TFLOPS, "algorithmic": flop}

    def hbm(nbytes, ms):
        a = nbytes / (ms * 1e-3) / 1e9
        return {"bound": "hbm", "achieved": a, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": a / HBM_PEAK_GBS, "algorithmic": nbytes}

    attn = mfma(work["attn_flop"], st["attn"])
    attn["hbm"] = hbm(work["attn_bytes"], st["attn"])
    return {"hash": mfma(work["hash_flop"], st["hash"]), "sort": hbm(work["sort_bytes"], st["sort"]),
            "attn": attn, "combine": hbm(work["combine_bytes"], st["combine"])}


def block_flop(wb: W.BlockWorkload) -> dict:
    """Algorithmic flops of one block direction (forward or inverse): the
    products of F (q and v projections, output projection: 3 x 2 M D D) and
    of G (2 x 2 M D d_ff), and the LSH attention's hash and chunk products."""
    M, D, F = wb.rows, wb.d_model, wb.d_ff
    att = W.Workload("block-attn", B=wb.B, H=wb.H, L=wb.L, d=64, dtype="bf16", n_buckets=wb.n_buckets,
                     n_rounds=wb.n_rounds, chunk=wb.chunk, causal=wb.causal)
    a = algorithmic_work(att)
    return {"proj": 3 * 2.0 * M * D * D, "ff": 2 * 2.0 * M * D * F, "hash": a["hash_flop"], "attn": a["attn_flop"]}


def run_block(wb: W.BlockWorkload, steps: int, warmup: int, cpu_budget: float) -> dict:
    """One step: the block forward (y1, y2 from x1, x2) and its inverse (x1, x2
    back from y1, y2), each one library call.  Also times F and G alone and
    the feed-forward's first product at one chunk's shape (M = ff_chunk,
    N = d_ff, K = d_model), the block's dominant kernel."""
    dev = torch.device("cuda:0")
    x = W.make_block_inputs(wb)

    def up(a):
        t = torch.from_numpy(np.ascontiguousarray(a))
        return (t.view(torch.int16).view(torch.bfloat16) if a.dtype == np.uint16 else t).to(dev)

    wts = lsh.BlockWeights(**{k: up(v) for k, v in x.items() if k not in ("x1", "x2")})
    cfg = lsh.BlockConfig.of(wb)
    x1, x2 = up(x["x1"]), up(x["x2"])
    y1, y2, r1, r2 = (torch.empty_like(x1) for _ in range(4))
    ws = torch.empty(lsh.block_workspace_bytes(cfg, lsh.LSH_BLOCK_OP_BLOCK), dtype=torch.uint8, device=dev)
    rows = wb.ff_chunk if 0 < wb.ff_chunk < wb.rows else wb.rows
    a = torch.randn((rows, wb.d_model), device=dev).to(torch.bfloat16)

    def timed(fn, n):
        for _ in range(warmup):
            fn()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record()
        for _ in range(n):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / n

    fwd = lambda: lsh.rev_block_fwd(cfg, wts, x1, x2, y1, y2, ws)
    inv = lambda: lsh.rev_block_inv(cfg, wts, y1, y2, r1, r2, ws)
    for _ in range(warmup):
        fwd()
        inv()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        fwd()
        inv()
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / steps
    res = {"ms_per_step": ms, "fwd_ms": timed(fwd, steps), "inv_ms": timed(inv, steps),
           "F_ms": timed(lambda: lsh.rev_attention(cfg, wts, x2, x1, 1.0, y1, ws), steps),
           "G_ms": timed(lambda: lsh.rev_feed_forward(cfg, wts, y1, x2, 1.0, y2, ws), steps),
           "ff1_ms": timed(lambda: lsh.linear_bf16(a, wts.w1, wts.b1, relu_bf16=True), steps)}
    fwd()
    inv()
    torch.cuda.synchronize()
    res["inverse_max_err"] = {"x1": float((r1 - x1).abs().max()), "x2": float((r2 - x2).abs().max())}
    if cpu_budget > 0:
        res["cpu_baseline"] = block_cpu_baseline(wb, cpu_budget)
    return res


def block_cpu_baseline(wb: W.BlockWorkload, budget_s: float) -> dict:
    """The oracle's block forward and inverse on a shortened sequence of the
    same block (same widths, heads and hashing), L halved until one pass
    should fit the budget; tokens/s of forward + inverse."""
    from oracle import block as OB  # test infrastructure: only for the reported baseline

    # flops of a forward + inverse per token: 2 x (3 projections 2 D^2 + 2
    # feed-forward products 2 D d_ff); fp64 NumPy products run at roughly
    # 20 GFLOP/s on the host
    per_token = 2 * (6 * wb.d_model ** 2 + 4 * wb.d_model * wb.d_ff)
    L = wb.L
    while L > 256 and L * per_token > budget_s * 20e9:
        L //= 2
    w = wb.scaled(L=L)
    x = W.make_block_inputs(w)
    f = lambda v: W.as_f64(v, "bf16") if v.dtype == np.uint16 else v.astype(np.float64)
    wh = OB.BlockWeights(**{k: f(v) for k, v in x.items() if k not in ("x1", "x2")})
    args = (wh, w.H, w.chunk, w.causal, w.ln_eps, w.ff_chunk)
    import oracle
    t0 = time.perf_counter()
    y1, y2 = OB.rev_block_fwd(x["x1"], x["x2"], *args)
    OB.rev_block_inv(y1, y2, *args)
    el = time.perf_counter() - t0
    return {"value": w.rows / el, "unit": "tokens/s", "cores": oracle.num_threads(), "kind": "oracle",
            "cpu_model": cpu_model(),
            "sample": f"one block forward and inverse at L={L} (B={w.B}, d_model={w.d_model}, d_ff={w.d_ff}, "
                      f"{w.H} heads, {w.n_rounds} rounds), fp64 NumPy and the C oracle, {el:.1f} s"}


def block_line(wb: W.BlockWorkload, steps: int, warmup: int, cpu_budget: float) -> dict:
    g = run_block(wb, steps, warmup, cpu_budget)
    fl = block_flop(wb)
    rows = wb.ff_chunk if 0 < wb.ff_chunk < wb.rows else wb.rows
    ff1 = 2.0 * rows * wb.d_model * wb.d_ff
    ach = ff1 / (g["ff1_ms"] * 1e-3) / 1e12
    total = sum(fl.values())
    line = {
        "metric": "reversible block (LSH attention + chunked feed-forward) forward + inverse tokens/sec",
        "value": wb.rows / (g["ms_per_step"] * 1e-3), "unit": "tokens/s", "n_gpus": 1, "steps": steps,
        "warmup": warmup, "ms_per_step": g["ms_per_step"], "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": wb.name, "B": wb.B, "L": wb.L, "H": wb.H, "d_model": wb.d_model, "d_ff": wb.d_ff,
                   "n_buckets": wb.n_buckets, "n_rounds": wb.n_rounds, "chunk": wb.chunk, "causal": wb.causal,
                   "ff_chunk": wb.ff_chunk},
        "stage_ms": {"forward": g["fwd_ms"], "inverse": g["inv_ms"], "F": g["F_ms"], "G": g["G_ms"]},
        "roofline": {"bound": "mfma", "achieved": ach, "peak": BF16_MFMA_PEAK_TFLOPS, "unit": "TFLOP/s",
                     "frac": ach / BF16_MFMA_PEAK_TFLOPS, "traffic": None, "stage": "ff1",
                     "kernels": ["gemm_bf16_kernel"], "algorithmic": ff1,
                     "shape": {"M": rows, "N": wb.d_ff, "K": wb.d_model}},
        "block_mfma_frac": total / (g["fwd_ms"] * 1e-3) / 1e12 / BF16_MFMA_PEAK_TFLOPS,
        "algorithmic_flop_per_direction": fl,
        "inverse_max_err": g["inverse_max_err"],
    }
    if "cpu_baseline" in g:
        line["cpu_baseline"] = g["cpu_baseline"]
    return line


SWEEP_LENGTHS = (1024, 2048, 4096, 8192, 16384, 32768, 65536)


def dense_flop(B: int, H: int, L: int, d: int, causal: bool) -> float:
    """Algorithmic flops of full attention: 2d for q.k and 2d for p*v per
    (query, key) pair that takes part (j <= i under causal masking)."""
    pairs = L * (L + 1) / 2 if causal else float(L) * L
    return 4.0 * d * pairs * B * H


def run_dense(B: int, H: int, L: int, q: torch.Tensor, v: torch.Tensor, causal: bool,
              steps: int, warmup: int) -> float:
    """Average ms of one dense attention forward (HIP events on the stream the
    kernels run on)."""
    cfg = lsh.Config(B=B, H=H, L=L, n_buckets=2, n_rounds=1, causal=causal)
    out = torch.empty_like(q)
    lse = torch.empty((B, H, L), dtype=torch.float32, device=q.device)
    ws = torch.empty(max(256, lsh.workspace_bytes(cfg, q.dtype, lsh.LSH_OP_DENSE_FWD)),
                     dtype=torch.uint8, device=q.device)
    for _ in range(warmup):
        lsh.lsh_dense_attn_fwd(cfg, q, v, out, lse, ws)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(steps):
        lsh.lsh_dense_attn_fwd(cfg, q, v, out, lse, ws)
    e1.record()
    torch.cuda.synchronize()
    if not torch.isfinite(out.float()).all():
        raise RuntimeError("non-finite dense output")
    return e0.elapsed_time(e1) / steps


def sweep_length(steps: int, warmup: int) -> None:
    """Speed against sequence length at a fixed number of tokens (the paper's
    speed-versus-length comparison, Sec. 5): the tokens and values of the
    64K x 16-head benchmark batch, cut into B = 65536/L sequences of length L.
    LSH attention: 8 rounds, chunks of 64, L/64 buckets (64 tokens per bucket on
    average, 1024 at 64K as in the benchmark); dense: full shared-QK attention.
    Both causal, bf16.  One JSON line per length."""
    base = W.WORKLOADS[W.HEADLINE]
    x = W.make_inputs(base)
    total, H, d = base.B * base.L, base.H, base.d
    dev = torch.device("cuda:0")
    for L in SWEEP_LENGTHS:
        B = total // L
        w = base.scaled(B=B, L=L, n_buckets=max(2, L // 64))
        q, v = (np.ascontiguousarray(t.reshape(H, B, L, d).transpose(1, 0, 2, 3))
                for t in (x["q"], x["v"]))
        rng = np.random.Generator(np.random.PCG64(L))
        R = rng.standard_normal((w.n_rounds, d, w.n_buckets // 2), dtype=np.float32)
        g = run_gpu(w, steps, warmup, {"q": q, "v": v, "R": R})
        qd = torch.from_numpy(q).view(torch.int16).view(torch.bfloat16).to(dev)
        vd = torch.from_numpy(v).view(torch.int16).view(torch.bfloat16).to(dev)
        dense_ms = run_dense(B, H, L, qd, vd, w.causal, steps, warmup)
        del qd, vd
        fl = dense_flop(B, H, L, d, w.causal)
        print(json.dumps({
            "sweep": "speed_vs_length", "L": L, "B": B, "H": H, "tokens": B * L,
            "n_buckets": w.n_buckets, "n_rounds": w.n_rounds, "causal": w.causal,
            "lsh_ms": g["ms_per_step"], "lsh_stage_ms": g["stage_ms"],
            "lsh_tokens_per_s": B * L / (g["ms_per_step"] * 1e-3),
            "dense_ms": dense_ms, "dense_tokens_per_s": B * L / (dense_ms * 1e-3),
            "dense_tflops": fl / (dense_ms * 1e-3) / 1e12,
            "dense_mfma_frac": fl / (dense_ms * 1e-3) / 1e12 / BF16_MFMA_PEAK_TFLOPS,
            "dense_over_lsh": dense_ms / g["ms_per_step"]}), flush=True)


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=50)
    ap.add_argument("--workload", default=W.HEADLINE, choices=sorted(W.WORKLOADS) + sorted(W.BLOCKS))
    ap.add_argument("--cpu-budget", type=float, default=8.0,
                    help="seconds of oracle time for the CPU baseline (0 to skip)")
    ap.add_argument("--copy-probe", type=int, default=0,
                    help="after timing, copy this many bytes device to device (a plain copy "
                         "kernel of known size, to scale HBM traffic counters)")
    ap.add_argument("--sweep-length", action="store_true",
                    help="instead of the benchmark line: LSH and dense attention speed at a "
                         "fixed number of tokens for L = 1K .. 64K (one JSON line per L)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only; --gpus {args.gpus} is not supported "
              "(each (batch, head) slice is independent; see the design notes for sharding)",
              file=sys.stderr)
        return 2
    if not torch.cuda.is_available():
        print("no GPU visible", file=sys.stderr)
        return 2
    lsh.lib()
    if args.workload in W.BLOCKS:
        print(json.dumps(block_line(W.BLOCKS[args.workload], args.steps, args.warmup, args.cpu_budget)), flush=True)
        return 0
    w = W.WORKLOADS[args.workload]
    if args.sweep_length:
        sweep_length(args.steps, args.warmup)
        return 0
    x = W.make_inputs(w)
    g = run_gpu(w, args.steps, args.warmup, x)
    if args.copy_probe > 0:
        n = args.copy_probe // 16 * 16
        src = torch.ones(n // 4, dtype=torch.int32, device="cuda:0")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    work = algorithmic_work(w)
    st = g["stage_ms"]
    # dominant stage: the one with the largest share of the step
    dom = max(st, key=st.get)
    spec = STAGES[dom]
    if spec["bound"] == "mfma":
        achieved = work[spec["work"]] / (st[dom] * 1e-3) / 1e12
        roof = {"bound": "mfma", "achieved": achieved, "peak": BF16_MFMA_PEAK_TFLOPS,
                "unit": "TFLOP/s"}
    else:
        achieved = work[spec["work"]] / (st[dom] * 1e-3) / 1e9
        roof = {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s"}
    roof["frac"] = roof["achieved"] / roof["peak"]
    roof["traffic"] = recorded_traffic(w.name, dom)
    roof["stage"] = dom
    roof["kernels"] = spec["kernels"]
    roof["algorithmic"] = work[spec["work"]]
    tokens = w.B * w.L
    value = tokens / (g["ms_per_step"] * 1e-3)
    line = {
        "metric": "LSH-attention fwd tokens/sec at L=64K, 8 rounds; % MFMA & HBM peak",
        "value": value, "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": g["ms_per_step"], "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": w.dtype, "data": "synthetic",
        "config": {"workload": w.name, "B": w.B, "H": w.H, "L": w.L, "d": w.d,
                   "n_buckets": w.n_buckets, "n_rounds": w.n_rounds, "chunk": w.chunk,
                   "causal": w.causal, "inputs": w.dist},
        "stage_ms": st,
        "roofline": roof,
        # every stage against its own roof, named (the dominant one is above)
        "rooflines": stage_rooflines(w, work, st),
    }
    if "bwd_ms" in g:
        # the backward (dq, dv) of the same batch, reported the same way
        bspec = STAGES["bwd"]
        bach = work["bwd_bytes"] / (g["bwd_ms"] * 1e-3) / 1e9
        line["backward"] = {
            "tokens_per_s": tokens / (g["bwd_wall_ms"] * 1e-3), "ms_per_step": g["bwd_wall_ms"],
            "kernel_ms": g["bwd_ms"],
            "roofline": {"bound": "hbm", "achieved": bach, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                         "frac": bach / HBM_PEAK_GBS,
                         "traffic": recorded_traffic(w.name, "bwd"), "stage": "bwd",
                         "kernels": bspec["kernels"], "algorithmic": work["bwd_bytes"]},
            "mfma_frac": work["bwd_flop"] / (g["bwd_ms"] * 1e-3) / 1e12 / BF16_MFMA_PEAK_TFLOPS,
        }
    if args.cpu_budget > 0:
        line["cpu_baseline"], line["parity"] = cpu_baseline(w, args.cpu_budget, x, g["state"])
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
