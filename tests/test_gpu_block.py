"""The reversible block on the GPU (include/lsh_block.h) against its oracle
(oracle/block.py, pinned in test_oracle_block.py): the product kernel against
float64 matrix products, the feed-forward layer G and the attention layer F
against the oracle, G's independence of the chunk size (bit for bit), and the
inverse reconstructing the block's inputs (Sec. 3, "RevNets").

Tolerances.  Both sides round the same product operands to bf16, so they
differ by the fp32 accumulation (about 1e-6 here) and by operands that land
on the other side of a bf16 rounding boundary (one bf16 unit, 2^-8 relative,
of an element; its effect on an output is that times a weight, ~1e-4).  G is
checked to 5e-3; F, whose attention output carries the attention's own bf16
tolerance, to 2e-2 (the attention's bound).  G's bound, 5e-3, is empirical:
the flips are rare and of random sign, and the errors measured are 1.6e-3
(d_ff = 256) and 2.7e-3 (d_ff = 4096, the benchmarked size); a rigorous
elementwise bound (every operand off by a unit) would be ~2^-8 |h| |W2|,
tens of times larger.  The product kernel itself is held to its rigorous
fp32 accumulation bound in test_linear_matches_float64_product.  F is run on the "exact" inputs
(rows of +-1 with balanced signs, projection weights k 2^-10), whose
LayerNorm and projections are exact in fp32 and fp64 alike, so both sides
hash identical q."""
import numpy as np
import pytest
import torch

from oracle import block as OB
from paper_2001_04451_amd import lsh
from paper_2001_04451_amd import workloads as W

from gpu_common import log

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    lsh.lib()
    return torch.device("cuda:0")


def _bf16(bits):
    return torch.from_numpy(np.ascontiguousarray(bits)).view(torch.int16).view(torch.bfloat16).cuda()


def _f32(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()


def _weights(x):
    dev = {k: (_bf16(v) if v.dtype == np.uint16 else _f32(v)) for k, v in x.items() if k not in ("x1", "x2")}
    host = OB.BlockWeights(**{k: (W.as_f64(v, "bf16") if v.dtype == np.uint16 else v.astype(np.float64))
                              for k, v in x.items() if k not in ("x1", "x2")})
    return lsh.BlockWeights(**dev), host


def _small(**kw):
    base = dict(B=2, L=320, H=2, d_ff=256, n_buckets=16, n_rounds=2, ff_chunk=0)
    base.update(kw)
    return W.BLOCKS["revblock_bf16_L65536"].scaled(**base)


@pytest.mark.parametrize("M,N,K", [(1000, 256, 192), (128, 128, 64), (77, 384, 1024)])
def test_linear_matches_float64_product(gpu, M, N, K):
    rng = np.random.default_rng(M + N + K)
    a = W.f32_to_bf16_bits(rng.standard_normal((M, K)).astype(np.float32))
    w = W.f32_to_bf16_bits((rng.standard_normal((N, K)) / np.sqrt(K)).astype(np.float32))
    bias = rng.standard_normal(N).astype(np.float32)
    resid = rng.standard_normal((M, N)).astype(np.float32)
    a64, w64 = W.as_f64(a, "bf16"), W.as_f64(w, "bf16")
    c = a64 @ w64.T + bias
    log("linear", M, N, K)
    got = lsh.linear_bf16(_bf16(a), _bf16(w), _f32(bias), _f32(resid), -1.0).cpu().numpy()
    # fp32 sums of K exact products: within K 2^-24 sum |a w| (plus the last roundings)
    bound = K * 2.0 ** -24 * (np.abs(a64) @ np.abs(w64).T + np.abs(bias)) + 2.0 ** -23 * (np.abs(resid) + np.abs(c))
    err = np.abs(got - (resid - c))
    assert (err <= bound).all(), f"max error {err.max()}, {(err > bound).sum()} over the bound"
    h = lsh.linear_bf16(_bf16(a), _bf16(w), _f32(bias), relu_bf16=True).float().cpu().numpy()
    want = OB.round_bf16(np.maximum(c, 0.0))
    # one bf16 unit where the fp32 sum lands across a rounding boundary
    assert (np.abs(h - want) <= 2.0 ** -7 * np.abs(want) + 1e-30).all()
    print(f"linear M={M} N={N} K={K}: max error {err.max():.2e}, bf16 outputs off by a unit: "
          f"{int((h != want).sum())} of {h.size}")


@pytest.mark.parametrize("ff_chunk", [0, 128, 250])
def test_feed_forward_matches_oracle(gpu, ff_chunk):
    w = _small(ff_chunk=ff_chunk)
    x = W.make_block_inputs(w)
    wd, wh = _weights(x)
    cfg = lsh.BlockConfig.of(w)
    y = np.random.default_rng(11).standard_normal((w.B, w.L, w.d_model)).astype(np.float32)
    log("feed-forward", ff_chunk)
    got = lsh.rev_feed_forward(cfg, wd, _f32(y)).cpu().numpy()
    want = OB.feed_forward(y.astype(np.float64), wh, w.ln_eps, ff_chunk)
    err = np.abs(got - want).max()
    print(f"feed-forward chunk={ff_chunk}: max-abs error {err:.2e} (|G| up to {np.abs(want).max():.2f})")
    assert err <= 5e-3


def test_feed_forward_chunks_bit_identical(gpu):
    """G's rows do not depend on how the rows are chunked (Sec. 3, "Chunking")."""
    w = _small()
    x = W.make_block_inputs(w)
    wd, _ = _weights(x)
    y = _f32(np.random.default_rng(12).standard_normal((w.B, w.L, w.d_model)))
    log("feed-forward chunks")
    outs = [lsh.rev_feed_forward(lsh.BlockConfig.of(w, ff_chunk=c), wd, y).cpu().numpy()
            for c in (0, 64, 100, 257, 640)]
    for o in outs[1:]:
        assert np.array_equal(o, outs[0])


@pytest.mark.parametrize("causal", [True, False])
def test_attention_layer_matches_oracle(gpu, causal):
    w = _small(exact=True, causal=causal)
    x = W.make_block_inputs(w)
    wd, wh = _weights(x)
    cfg = lsh.BlockConfig.of(w)
    log("attention layer", causal)
    f = lsh.rev_attention(cfg, wd, _f32(x["x2"])).cpu().numpy()
    want = OB.attention_layer(x["x2"].astype(np.float64), wh, w.H, w.chunk, causal, w.ln_eps)
    err = np.abs(f - want).max()
    print(f"attention layer causal={causal}: max-abs error {err:.2e} (|F| up to {np.abs(want).max():.2f})")
    assert err <= 2e-2
    # with a residual and the inverse's sign
    r = np.random.default_rng(13).standard_normal(x["x2"].shape).astype(np.float32)
    g = lsh.rev_attention(cfg, wd, _f32(x["x2"]), _f32(r), -1.0).cpu().numpy()
    assert np.abs(g - (r - want)).max() <= 2e-2 + 1e-6


def _rounding(*ts):
    """Two fp32 roundings of the largest magnitude involved (an fp32 sum and
    its exact undoing reproduce a value to that)."""
    return 2.0 ** -22 * np.maximum.reduce([np.abs(t) for t in ts]) + 1e-30


def test_block_forward_and_inverse(gpu):
    """y1 against the oracle, the block's wiring bit for bit (y1 = x1 + F(x2)
    and y2 = x2 + G(y1) with the library's own F and G, one fp32 rounding
    each), then the inverse on the GPU reproducing x1 and x2 to the rounding
    of the fp32 residual additions.  With x2 rows of +-1 the inverse's
    LayerNorm sees x2 up to that rounding, which leaves its bf16 outputs,
    hence F(x2), unchanged."""
    w = _small(exact=True, ff_chunk=200)
    x = W.make_block_inputs(w)
    wd, wh = _weights(x)
    cfg = lsh.BlockConfig.of(w)
    log("block forward and inverse")
    x1, x2 = _f32(x["x1"]), _f32(x["x2"])
    y1, y2 = lsh.rev_block_fwd(cfg, wd, x1, x2)
    r1, r2 = lsh.rev_block_inv(cfg, wd, y1, y2)
    f = lsh.rev_attention(cfg, wd, x2).cpu().numpy()
    g = lsh.rev_feed_forward(cfg, wd, y1).cpu().numpy()
    y1, y2, r1, r2 = (t.cpu().numpy() for t in (y1, y2, r1, r2))
    assert np.array_equal(y1, x["x1"] + f) and np.array_equal(y2, x["x2"] + g)
    o1, _ = OB.rev_block_fwd(x["x1"], x["x2"], wh, w.H, w.chunk, w.causal, w.ln_eps, w.ff_chunk)
    e1 = np.abs(y1 - o1).max()
    d1, d2 = np.abs(r1 - x["x1"]), np.abs(r2 - x["x2"])
    print(f"block: forward error y1 {e1:.2e}; inverse error x1 {d1.max():.2e} x2 {d2.max():.2e}")
    assert e1 <= 2e-2
    assert (d2 <= _rounding(y2, x["x2"])).all()
    assert (d1 <= _rounding(y1, x["x1"])).all()


def test_block_inverse_general_inputs(gpu):
    """Gaussian x1 and x2: x2 comes back to rounding everywhere (G(y1) is
    recomputed from the same y1); x1 wherever F(x2') rounds its operands as
    F(x2) did.  A LayerNorm output of x2' may land on the other side of a
    bf16 rounding boundary and move q by a bf16 unit, which can move a
    near-tie row to another bucket: then x1 differs by F's change.  Such rows
    must be rare."""
    w = _small(L=512)
    x = W.make_block_inputs(w)
    wd, _ = _weights(x)
    cfg = lsh.BlockConfig.of(w)
    log("block inverse, general inputs")
    y1, y2 = lsh.rev_block_fwd(cfg, wd, _f32(x["x1"]), _f32(x["x2"]))
    r1, r2 = lsh.rev_block_inv(cfg, wd, y1, y2)
    y1, y2, r1, r2 = (t.cpu().numpy() for t in (y1, y2, r1, r2))
    assert (np.abs(r2 - x["x2"]) <= _rounding(y2, x["x2"])).all()
    exact = (np.abs(r1 - x["x1"]) <= _rounding(y1, x["x1"])).all(axis=-1)
    close = (np.abs(r1 - x["x1"]) <= 1e-2).all(axis=-1)
    print(f"general inputs: rows reconstructed to rounding {exact.mean():.4f}, within 1e-2 {close.mean():.4f}")
    assert exact.mean() >= 0.8 and close.mean() >= 0.99


def test_full_size_block(gpu):
    """The block at the benchmarked size (L = 65536, d_model = 1024, d_ff =
    4096, 16 heads, 8 rounds of 1024 buckets, feed-forward chunks of 16384
    rows) on exact inputs: G on 64 sampled rows against the oracle, and the
    inverse reconstructing x1 and x2 everywhere."""
    w = W.BLOCKS["revblock_bf16_L65536"].scaled(exact=True)
    x = W.make_block_inputs(w)
    wd, wh = _weights(x)
    cfg = lsh.BlockConfig.of(w)
    log("full-size block")
    x1, x2 = _f32(x["x1"]), _f32(x["x2"])
    y1, y2 = lsh.rev_block_fwd(cfg, wd, x1, x2)
    r1, r2 = lsh.rev_block_inv(cfg, wd, y1, y2)
    g = (y2 - x2)  # G(y1) up to one fp32 rounding
    rows = np.sort(np.random.default_rng(14).choice(w.L, 64, replace=False))
    y1s = y1[0, rows].cpu().numpy().astype(np.float64)
    want = OB.feed_forward(y1s, wh, w.ln_eps)
    err = np.abs(g[0, rows].cpu().numpy() - want).max()
    d1 = (r1 - x1).abs().max().item()
    d2 = (r2 - x2).abs().max().item()
    print(f"full size: G on sampled rows max-abs error {err:.2e}; inverse error x1 {d1:.2e} x2 {d2:.2e}")
    assert err <= 5e-3
    b1 = float(torch.maximum(y1.abs(), x1.abs()).max()) * 2.0 ** -22
    b2 = float(torch.maximum(y2.abs(), x2.abs()).max()) * 2.0 ** -22
    assert d1 <= b1 and d2 <= b2
