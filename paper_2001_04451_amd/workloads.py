"""Seeded synthetic inputs for LSH attention, shared by the tests, the bench
and the oracle checks.

This module holds no arithmetic of the method: it only draws random numbers,
rounds fp32 draws to bf16 and names the workloads.  The paper's own data
(enwik8-64K at L = 65536, imagenet64 at L = 12288; Sec. 5) is not available,
so Gaussian and Gaussian-mixture inputs with the paper's sequence lengths and
head width stand in for it.

Draw order, from one ``numpy.random.Generator(PCG64(seed))``:
  1. R  [n_rounds, d, n_buckets/2] fp32, iid N(0, 1);
  2. Q  [B, H, L, d]: iid N(0, 1), or a mixture (per (b, h): centres
     [K, d] ~ N(0, 1), then component labels [L] ~ U{0..K-1}, then noise
     [L, d] ~ N(0, 1) scaled by sigma; q = centre[label] + sigma * noise);
  3. V  [B, H, L, d], iid N(0, 1);
  4. dO [B, H, L, d], iid N(0, 1) (only for workloads with a backward).
bf16 tensors are fp32 draws rounded to nearest even and are carried as their
uint16 bit patterns.

The reversible-block workloads (BLOCKS, make_block_inputs) draw, in order:
R; x1 [B, L, d_model] ~ N(0, 1); x2 the same, or for "exact" inputs rows of
+-1 with d_model/2 of each sign in random order; LayerNorm 1 gain 1 + 0.1 N
and bias 0.1 N (exact inputs: 1 and 0); W_qk and W_v [H*64, d_model] ~
N(0, 1/d_model) in bf16 (exact inputs: k 2^-10 with k uniform in -127..127);
W_o [d_model, H*64] ~ N(0, 1/(H*64)); LayerNorm 2 like LayerNorm 1 (always
random); W1 [d_ff, d_model] ~ N(0, 1/d_model), b1 [d_ff] ~ 0.1 N;
W2 [d_model, d_ff] ~ N(0, 1/d_ff), b2 [d_model] ~ 0.1 N.  Weight matrices
are bf16 bit patterns, the rest fp32.
"""
from __future__ import annotations

from dataclasses import dataclass, field, replace

import numpy as np


@dataclass(frozen=True)
class Workload:
    name: str
    B: int
    H: int
    L: int
    d: int
    dtype: str  # "f32" or "bf16"
    n_buckets: int
    n_rounds: int
    chunk: int
    causal: bool
    dist: str = "iid"  # "iid" or "mixture"
    n_components: int = 0
    sigma: float = 0.3
    seed: int = 0
    backward: bool = False
    notes: str = field(default="", compare=False)

    @property
    def rows(self) -> int:
        return self.B * self.H * self.L

    @property
    def row_rounds(self) -> int:
        return self.rows * self.n_rounds

    def scaled(self, **kw) -> "Workload":
        return replace(self, **kw)


# The five workloads: shapes, dtypes, hashing parameters and input structure.
WORKLOADS = {
    "tiny_f32_L1024": Workload(
        "tiny_f32_L1024", B=1, H=1, L=1024, d=64, dtype="f32", n_buckets=16, n_rounds=1,
        chunk=64, causal=False, dist="iid", seed=0,
        notes="fp32, iid queries, one round"),
    "mixture_bf16_L4096": Workload(
        "mixture_bf16_L4096", B=4, H=8, L=4096, d=64, dtype="bf16", n_buckets=64, n_rounds=2,
        chunk=64, causal=False, dist="mixture", n_components=32, sigma=0.3, seed=1,
        notes="32-Gaussian mixture: uneven buckets"),
    "causal_bf16_L16384": Workload(
        "causal_bf16_L16384", B=2, H=8, L=16384, d=64, dtype="bf16", n_buckets=256, n_rounds=4,
        chunk=64, causal=True, dist="iid", seed=2,
        notes="causal with self-mask fallback"),
    "long_bf16_L65536": Workload(
        "long_bf16_L65536", B=1, H=16, L=65536, d=64, dtype="bf16", n_buckets=1024, n_rounds=8,
        chunk=64, causal=True, dist="mixture", n_components=256, sigma=0.3, seed=3,
        notes="d_model 1024 as 16 heads of 64; 256-Gaussian mixture"),
    "fwdbwd_bf16_L32768": Workload(
        "fwdbwd_bf16_L32768", B=8, H=8, L=32768, d=64, dtype="bf16", n_buckets=512, n_rounds=4,
        chunk=64, causal=True, dist="iid", seed=4, backward=True,
        notes="forward and backward (dq, dv)"),
}

# The workload the headline throughput figure is quoted on.
HEADLINE = "long_bf16_L65536"


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 to the nearest bf16 (ties to even); returns uint16 bit patterns.
    Infinities stay infinite and NaNs stay (quiet) NaNs."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = (b >> 16) & np.uint32(1)
    r += np.uint32(0x7FFF)
    r += b  # no wrap-around: a finite value's bits are at most 0xFF7FFFFF
    r >>= 16
    special = (b & np.uint32(0x7F800000)) == np.uint32(0x7F800000)
    if special.any():
        hi = b[special] >> 16
        r[special] = np.where((b[special] & np.uint32(0x7FFFFF)) != 0, hi | np.uint32(0x40), hi)
    return r.astype(np.uint16)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to fp32."""
    return (np.ascontiguousarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def _draw_q(rng: np.random.Generator, w: Workload) -> np.ndarray:
    if w.dist == "iid":
        return rng.standard_normal((w.B, w.H, w.L, w.d), dtype=np.float32)
    if w.dist == "mixture":
        K = w.n_components
        centres = rng.standard_normal((w.B, w.H, K, w.d), dtype=np.float32)
        labels = rng.integers(0, K, size=(w.B, w.H, w.L))
        noise = rng.standard_normal((w.B, w.H, w.L, w.d), dtype=np.float32)
        bi = np.arange(w.B)[:, None, None]
        hi = np.arange(w.H)[None, :, None]
        q = centres[bi, hi, labels]
        q += np.float32(w.sigma) * noise
        return q
    raise ValueError(f"unknown distribution {w.dist!r}")


def make_inputs(w: Workload, seed: int | None = None, with_dout: bool | None = None) -> dict:
    """Draw R, q, v (and dout) for workload ``w``.

    Returns a dict of NumPy arrays: ``R`` fp32; ``q``, ``v`` and ``dout`` as
    fp32 (dtype "f32") or as uint16 bf16 bit patterns (dtype "bf16").
    """
    rng = np.random.Generator(np.random.PCG64(w.seed if seed is None else seed))
    R = rng.standard_normal((w.n_rounds, w.d, w.n_buckets // 2), dtype=np.float32)
    q = _draw_q(rng, w)
    v = rng.standard_normal((w.B, w.H, w.L, w.d), dtype=np.float32)
    out = {"R": R}
    if with_dout is None:
        with_dout = w.backward
    dout = rng.standard_normal((w.B, w.H, w.L, w.d), dtype=np.float32) if with_dout else None
    if w.dtype == "bf16":
        out["q"] = f32_to_bf16_bits(q)
        out["v"] = f32_to_bf16_bits(v)
        if dout is not None:
            out["dout"] = f32_to_bf16_bits(dout)
    elif w.dtype == "f32":
        out["q"], out["v"] = q, v
        if dout is not None:
            out["dout"] = dout
    else:
        raise ValueError(f"unknown dtype {w.dtype!r}")
    return out


@dataclass(frozen=True)
class BlockWorkload:
    """A reversible block (attention half + chunked feed-forward half) around
    LSH attention with H heads of 64 (d_model = 64 H)."""
    name: str
    B: int
    L: int
    H: int
    d_ff: int
    n_buckets: int
    n_rounds: int
    chunk: int
    causal: bool
    ff_chunk: int           # rows per feed-forward chunk (0: all rows)
    ln_eps: float = 1e-5
    seed: int = 0
    exact: bool = False     # inputs whose LayerNorm and projections are exact
    notes: str = field(default="", compare=False)

    @property
    def d_model(self) -> int:
        return 64 * self.H

    @property
    def rows(self) -> int:
        return self.B * self.L

    def scaled(self, **kw) -> "BlockWorkload":
        return replace(self, **kw)


BLOCKS = {
    "revblock_bf16_L65536": BlockWorkload(
        "revblock_bf16_L65536", B=1, L=65536, H=16, d_ff=4096, n_buckets=1024, n_rounds=8, chunk=64,
        causal=True, ff_chunk=16384, seed=5,
        notes="d_model 1024, d_ff 4096 (the paper's sizes), the long workload's attention"),
}


def make_block_inputs(w: BlockWorkload, seed: int | None = None) -> dict:
    """Draw R, x1, x2 and the block's weights (see the module notes)."""
    rng = np.random.Generator(np.random.PCG64(w.seed if seed is None else seed))
    D, F, HD = w.d_model, w.d_ff, 64 * w.H
    out = {"R": rng.standard_normal((w.n_rounds, 64, w.n_buckets // 2), dtype=np.float32)}
    out["x1"] = rng.standard_normal((w.B, w.L, D), dtype=np.float32)
    if w.exact:
        signs = np.tile(np.repeat(np.array([1.0, -1.0], np.float32), D // 2), (w.B * w.L, 1))
        out["x2"] = rng.permuted(signs, axis=1).reshape(w.B, w.L, D)
    else:
        out["x2"] = rng.standard_normal((w.B, w.L, D), dtype=np.float32)

    def ln_params(unit):
        if unit:
            return np.ones(D, np.float32), np.zeros(D, np.float32)
        g = (1.0 + 0.1 * rng.standard_normal(D)).astype(np.float32)
        return g, (0.1 * rng.standard_normal(D)).astype(np.float32)

    def dense(rows, cols, fan_in):
        return f32_to_bf16_bits((rng.standard_normal((rows, cols)) / np.sqrt(fan_in)).astype(np.float32))

    out["ln1_g"], out["ln1_b"] = ln_params(w.exact)
    if w.exact:
        k = rng.integers(-127, 128, size=(2, HD, D))
        out["w_qk"] = f32_to_bf16_bits((k[0] * 2.0 ** -10).astype(np.float32))
        out["w_v"] = f32_to_bf16_bits((k[1] * 2.0 ** -10).astype(np.float32))
    else:
        out["w_qk"] = dense(HD, D, D)
        out["w_v"] = dense(HD, D, D)
    out["w_o"] = dense(D, HD, HD)
    out["ln2_g"], out["ln2_b"] = ln_params(False)
    out["w1"] = dense(F, D, D)
    out["b1"] = (0.1 * rng.standard_normal(F)).astype(np.float32)
    out["w2"] = dense(D, F, F)
    out["b2"] = (0.1 * rng.standard_normal(D)).astype(np.float32)
    return out


def as_f64(x: np.ndarray, dtype: str) -> np.ndarray:
    """Exact float64 values of an input tensor carried as fp32 or bf16 bits."""
    if dtype == "bf16":
        return bf16_bits_to_f32(x).astype(np.float64)
    return np.asarray(x, dtype=np.float32).astype(np.float64)
