"""Pins of the reversible-block oracle (oracle/block.py) against what the
paper and the mathematics fix, independent of the GPU library:

* LayerNorm and the feed-forward layer against PyTorch's own layer_norm,
  linear and relu (float64);
* the bf16 rounding against the bit-level fp32 -> bf16 rounding of the input
  generator and against hand-built ties;
* the attention layer, with identity projections, against the LSH attention
  oracle run on the normalised rows, per head (the head split and merge);
* chunked feed-forward equal to the unchunked one (Sec. 3, "Chunking");
* the block's inverse reconstructing its inputs (Sec. 3, "RevNets"), and
  the block reducing to the identity when both residual branches are zero.
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as Fn

import oracle
from oracle import block as OB
from paper_2001_04451_amd import workloads as W


def _weights(x, w):
    f = lambda k: W.as_f64(x[k], "bf16") if x[k].dtype == np.uint16 else x[k].astype(np.float64)
    return OB.BlockWeights(**{k: f(k) for k in ("ln1_g", "ln1_b", "w_qk", "w_v", "w_o", "ln2_g", "ln2_b",
                                                 "w1", "b1", "w2", "b2")}, R=x["R"].astype(np.float64))


def _small(**kw):
    base = dict(B=2, L=256, H=2, d_ff=256, n_buckets=8, n_rounds=2, ff_chunk=96)
    base.update(kw)
    return W.BLOCKS["revblock_bf16_L65536"].scaled(**base)


def test_layer_norm_matches_torch():
    rng = np.random.default_rng(1)
    x = rng.standard_normal((5, 7, 96)) * 3 + 1
    g, b = rng.standard_normal(96), rng.standard_normal(96)
    want = Fn.layer_norm(torch.from_numpy(x), (96,), torch.from_numpy(g), torch.from_numpy(b), eps=1e-5)
    np.testing.assert_allclose(OB.layer_norm(x, g, b, 1e-5), want.numpy(), rtol=0, atol=1e-12)


def test_round_bf16():
    rng = np.random.default_rng(2)
    x = (rng.standard_normal(20000) * np.exp(rng.uniform(-30, 30, 20000))).astype(np.float32)
    x[:8] = [0.0, -0.0, 1.0, -2.5, 3e-39, -1e-40, 65504.0, 1e30]  # zero, exact, subnormal
    want = W.bf16_bits_to_f32(W.f32_to_bf16_bits(x)).astype(np.float64)
    np.testing.assert_array_equal(OB.round_bf16(x.astype(np.float64)), want)
    # ties to even: 1 + 2^-8 lies halfway between 1 and 1 + 2^-7
    np.testing.assert_array_equal(OB.round_bf16(np.array([1 + 2.0 ** -8, 1 + 3 * 2.0 ** -8])),
                                  [1.0, 1 + 2.0 ** -6])


def test_feed_forward_matches_torch():
    w = _small()
    x = W.make_block_inputs(w)
    wt = _weights(x, w)
    y = np.random.default_rng(3).standard_normal((2, 40, w.d_model))
    t = lambda a: torch.from_numpy(np.asarray(a, np.float64))
    n = OB.round_bf16(Fn.layer_norm(t(y), (w.d_model,), t(wt.ln2_g), t(wt.ln2_b), eps=w.ln_eps).numpy())
    h = OB.round_bf16(Fn.relu(Fn.linear(t(n), t(wt.w1), t(wt.b1))).numpy())
    want = Fn.linear(t(h), t(wt.w2), t(wt.b2)).numpy()
    np.testing.assert_allclose(OB.feed_forward(y, wt, w.ln_eps), want, rtol=0, atol=1e-10)


@pytest.mark.parametrize("chunk_rows", [1, 7, 33, 80, 1000])
def test_feed_forward_chunks(chunk_rows):
    w = _small()
    wt = _weights(W.make_block_inputs(w), w)
    y = np.random.default_rng(4).standard_normal((2, 40, w.d_model))
    np.testing.assert_allclose(OB.feed_forward(y, wt, w.ln_eps, chunk_rows), OB.feed_forward(y, wt, w.ln_eps),
                               rtol=0, atol=1e-12)


@pytest.mark.parametrize("heads", [1, 2])
def test_attention_layer_identity_projections(heads):
    """With W_qk = W_v = W_o = I, LayerNorm gain 1 and bias 0, F(x) is the LSH
    attention of the (bf16-rounded) normalised rows, head h taking columns
    64h .. 64h+63."""
    D = 64 * heads
    rng = np.random.default_rng(5 + heads)
    x = rng.standard_normal((2, 128, D))
    R = rng.standard_normal((2, 64, 4))
    eye = np.eye(D)
    wt = OB.BlockWeights(ln1_g=np.ones(D), ln1_b=np.zeros(D), w_qk=eye, w_v=eye, w_o=eye, R=R,
                         ln2_g=None, ln2_b=None, w1=None, b1=None, w2=None, b2=None)
    got = OB.attention_layer(x, wt, heads, chunk=32, causal=True, ln_eps=1e-5)
    n = OB.round_bf16(OB.layer_norm(x, np.ones(D), np.zeros(D), 1e-5))
    for h in range(heads):
        qh = n[:, :, 64 * h:64 * h + 64][:, None].copy()       # [B, 1, L, 64]
        want = oracle.lsh_attention_fwd(qh, qh, R, 32, True)["out"][:, 0]
        np.testing.assert_allclose(got[:, :, 64 * h:64 * h + 64], OB.round_bf16(want), rtol=0, atol=1e-12)


def test_block_inverse_reconstructs():
    w = _small()
    x = W.make_block_inputs(w)
    wt = _weights(x, w)
    x1, x2 = x["x1"].astype(np.float64), x["x2"].astype(np.float64)
    args = (wt, w.H, w.chunk, w.causal, w.ln_eps, w.ff_chunk)
    y1, y2 = OB.rev_block_fwd(x1, x2, *args)
    assert np.abs(y1 - x1).max() > 1e-2 and np.abs(y2 - x2).max() > 1e-2  # the branches do something
    r1, r2 = OB.rev_block_inv(y1, y2, *args)
    assert np.abs(r2 - x2).max() < 1e-12
    assert np.abs(r1 - x1).max() < 1e-12


def test_block_with_zero_branches_is_identity():
    w = _small()
    x = W.make_block_inputs(w)
    wt = _weights(x, w)
    wt.w_o = np.zeros_like(wt.w_o)
    wt.w2, wt.b2 = np.zeros_like(wt.w2), np.zeros_like(wt.b2)
    y1, y2 = OB.rev_block_fwd(x["x1"], x["x2"], wt, w.H, w.chunk, w.causal, w.ln_eps, w.ff_chunk)
    np.testing.assert_array_equal(y1, x["x1"].astype(np.float64))
    np.testing.assert_array_equal(y2, x["x2"].astype(np.float64))


def test_exact_inputs_are_exact():
    """The "exact" block inputs: LayerNorm of a +-1 row with balanced signs is
    +-1/sqrt(1 + eps), which rounds to +-1 in bf16, and the projections are
    sums of k 2^-10 with |k| < 128 over d_model terms, integers times 2^-10
    below 2^24 in magnitude: exact in fp32 as in fp64."""
    w = _small(exact=True)
    x = W.make_block_inputs(w)
    wt = _weights(x, w)
    n = OB.round_bf16(OB.layer_norm(x["x2"], wt.ln1_g, wt.ln1_b, w.ln_eps))
    assert set(np.unique(n)) == {-1.0, 1.0}
    q = n @ wt.w_qk.T
    assert np.array_equal(q.astype(np.float32).astype(np.float64), q)
    assert np.abs(q * 2 ** 10).max() < 2 ** 24 and np.array_equal(np.rint(q * 2 ** 10), q * 2 ** 10)
