"""CPU oracle of the reversible block around LSH attention (Reformer Sec. 3,
"RevNets", "Reversible Transformer" and "Chunking").

TEST INFRASTRUCTURE ONLY, like the rest of this package: only the test suite,
``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of ``bench.py`` may
use it.  Plain NumPy in float64, written from the paper's equations:

* RevNet block: y1 = x1 + F(x2), y2 = x2 + G(y1); inverse by subtracting the
  residuals in the opposite order: x2 = y2 - G(y1), x1 = y1 - F(x2) (Sec. 3,
  "RevNets", the pair of equations and eq. reverse-ff).
* F is the attention layer and G the feed-forward layer, each with its
  layer normalisation inside the residual branch (Sec. 3, "Reversible
  Transformer"): F(x) = Attention(LayerNorm(x)), G(x) = FeedForward(LayerNorm(x)).
* The attention layer is shared-QK LSH attention (Sec. 2): one projection
  gives the queries (the keys are the normalised queries), another the
  values, split into heads of 64; the heads' outputs are concatenated and
  projected back to d_model.
* The feed-forward layer is applied to chunks of positions, one after
  another (Sec. 3, "Chunking", the equation for Y2): the result does not
  depend on the chunk size.

Readings where the paper is silent (also listed in the design notes):
* The feed-forward activation is ReLU (the Transformer's).
* Every matrix product of the block takes bf16 operands (the weights are
  bf16): the normalised rows, q and v, the attention's output and the
  feed-forward's hidden layer are rounded to bf16 (nearest, ties to even)
  where they enter a product.  The rounding of q decides bucket ids, so the
  oracle takes these roundings too; all arithmetic stays in float64.
* Chunks run over the flattened (batch, position) rows.

Layouts (row-major, like the C ABI): x [B, L, d_model]; W_qk and W_v
[H*64, d_model]; W_o [d_model, H*64]; W1 [d_ff, d_model], b1 [d_ff];
W2 [d_model, d_ff], b2 [d_model]; LayerNorm gains and biases [d_model].
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from . import lsh_attention_fwd


@dataclass
class BlockWeights:
    ln1_g: np.ndarray
    ln1_b: np.ndarray
    w_qk: np.ndarray
    w_v: np.ndarray
    w_o: np.ndarray
    R: np.ndarray
    ln2_g: np.ndarray
    ln2_b: np.ndarray
    w1: np.ndarray
    b1: np.ndarray
    w2: np.ndarray
    b2: np.ndarray


def layer_norm(x, g, b, eps):
    """(x - mean) / sqrt(var + eps) * g + b over the last axis (biased variance)."""
    x = np.asarray(x, np.float64)
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + eps) * np.asarray(g, np.float64) + np.asarray(b, np.float64)


def round_bf16(x):
    """Nearest bf16 value (ties to even) of float64 values, as float64.
    bf16 keeps 8 significant bits over fp32's exponent range; values whose
    leading bit lies below 2^-126 keep fewer (subnormals)."""
    x = np.asarray(x, np.float64)
    out = x.copy()
    fin = np.isfinite(x) & (x != 0)
    _, k = np.frexp(x[fin])                     # |x| in [2^(k-1), 2^k)
    quantum = np.ldexp(1.0, np.maximum(k - 1, -126) - 7)
    out[fin] = np.rint(x[fin] / quantum) * quantum
    return out


def attention_layer(x, w: BlockWeights, heads, chunk, causal, ln_eps, scale=None):
    """F(x) = Attention(LayerNorm(x)) for x [B, L, d_model]; product operands
    rounded to bf16."""
    B, L, D = x.shape
    n = round_bf16(layer_norm(x, w.ln1_g, w.ln1_b, ln_eps))
    q = round_bf16(n @ np.asarray(w.w_qk, np.float64).T)
    v = round_bf16(n @ np.asarray(w.w_v, np.float64).T)
    # [B, L, H*64] -> [B, H, L, 64]
    q = q.reshape(B, L, heads, 64).transpose(0, 2, 1, 3).copy()
    v = v.reshape(B, L, heads, 64).transpose(0, 2, 1, 3).copy()
    r = lsh_attention_fwd(q, v, np.asarray(w.R, np.float64), chunk, causal, scale)
    o = round_bf16(r["out"]).transpose(0, 2, 1, 3).reshape(B, L, heads * 64)
    return o @ np.asarray(w.w_o, np.float64).T


def feed_forward(x, w: BlockWeights, ln_eps, chunk_rows=0):
    """G(x) = relu(LayerNorm(x) W1^T + b1) W2^T + b2, computed chunk by chunk
    over the flattened rows (chunk_rows <= 0: all rows at once); product
    operands rounded to bf16."""
    shape = x.shape
    rows = np.asarray(x, np.float64).reshape(-1, shape[-1])
    c = rows.shape[0] if chunk_rows <= 0 else chunk_rows
    w1, w2 = np.asarray(w.w1, np.float64), np.asarray(w.w2, np.float64)
    parts = []
    for s in range(0, rows.shape[0], c):
        n = round_bf16(layer_norm(rows[s:s + c], w.ln2_g, w.ln2_b, ln_eps))
        h = round_bf16(np.maximum(n @ w1.T + np.asarray(w.b1, np.float64), 0.0))
        parts.append(h @ w2.T + np.asarray(w.b2, np.float64))
    return np.concatenate(parts, axis=0).reshape(shape[:-1] + (w2.shape[0],))


def rev_block_fwd(x1, x2, w: BlockWeights, heads, chunk, causal, ln_eps, ff_chunk=0):
    """(y1, y2) = (x1 + F(x2), x2 + G(y1))."""
    y1 = np.asarray(x1, np.float64) + attention_layer(x2, w, heads, chunk, causal, ln_eps)
    y2 = np.asarray(x2, np.float64) + feed_forward(y1, w, ln_eps, ff_chunk)
    return y1, y2


def rev_block_inv(y1, y2, w: BlockWeights, heads, chunk, causal, ln_eps, ff_chunk=0):
    """(x1, x2) from (y1, y2): x2 = y2 - G(y1), then x1 = y1 - F(x2)."""
    x2 = np.asarray(y2, np.float64) - feed_forward(y1, w, ln_eps, ff_chunk)
    x1 = np.asarray(y1, np.float64) - attention_layer(x2, w, heads, chunk, causal, ln_eps)
    return x1, x2
