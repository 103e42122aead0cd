"""Shared helpers of the GPU parity tests (imported by test_gpu_*.py)."""
from __future__ import annotations

import sys

import numpy as np
import torch

from paper_2001_04451_amd import workloads as W


def log(*args) -> None:
    """Name the case before every GPU step, flushed, so a fault is attributable."""
    print("[gpu-case]", *args, flush=True)
    sys.stdout.flush()


def to_device(x: np.ndarray, dtype: str) -> torch.Tensor:
    """Upload generator output: bf16 bit patterns become torch.bfloat16."""
    t = torch.from_numpy(np.ascontiguousarray(x))
    if dtype == "bf16":
        t = t.view(torch.int16).view(torch.bfloat16)
    return t.cuda()


def torch_dtype(dtype: str) -> torch.dtype:
    return torch.bfloat16 if dtype == "bf16" else torch.float32


def out_tolerance(dtype: str) -> float:
    """Max-abs output error allowed against the fp64 oracle: 1e-5 for fp32
    inputs, 2e-2 for bf16 inputs with fp32 accumulation."""
    return 1e-5 if dtype == "f32" else 2e-2


def rounds_f64(o_rounds: torch.Tensor, o_exp: torch.Tensor | None) -> np.ndarray:
    """Per-round outputs as float64: fp32 rows as they are; fp16 rows times
    2^o_exp (the scale lsh_chunk_attn_fwd applies to bf16 calls)."""
    o = o_rounds.float().cpu().numpy().astype(np.float64)
    if o_exp is None:
        return o
    return np.ldexp(o, o_exp.cpu().numpy().astype(np.int32)[..., None])


def lse_close(gpu: np.ndarray, ref: np.ndarray, dtype: str) -> np.ndarray:
    """Log-partition comparison.  Rows whose only target is themselves sit at
    z ~ -1e5, where one fp32 spacing is 2^-7, so the bound is relative there."""
    abs_tol = 1e-5 if dtype == "f32" else 2e-2
    return np.abs(gpu - ref) <= abs_tol + 2e-7 * np.abs(ref)


def small(name: str, **kw) -> W.Workload:
    """A reduced copy of a named workload (same hashing parameters, dtype and
    input structure) that the oracle finishes in seconds."""
    return W.WORKLOADS[name].scaled(**kw)
