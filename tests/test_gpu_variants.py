"""Variants of the method the paper does not spell out, on the GPU against the
oracle (which is pinned for each of them in test_oracle_pins.py): a
look-ahead chunk, attention across buckets, chunks of 128 and one R per head.
Whole forwards on seeded inputs; bucket ids and permutations bit for bit,
outputs within 1e-5 (fp32) or 2e-2 (bf16) max-abs."""
import numpy as np
import pytest
import torch

import oracle
from paper_2001_04451_amd import lsh
from paper_2001_04451_amd import workloads as W

from gpu_common import log, lse_close, out_tolerance, small, to_device

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    lsh.lib()
    return torch.device("cuda:0")


def _forward(w, R, cfg, after=0, across=False):
    x = W.make_inputs(w)
    q64, v64 = W.as_f64(x["q"], w.dtype), W.as_f64(x["v"], w.dtype)
    ref = oracle.lsh_attention_fwd(q64, v64, R.astype(np.float64), w.chunk, w.causal,
                                   after=after, across=across)
    st = lsh.lsh_attention_fwd(cfg, to_device(x["q"], w.dtype), to_device(x["v"], w.dtype),
                               to_device(R, "f32"))
    torch.cuda.synchronize()
    assert np.array_equal(st.buckets.cpu().numpy(), ref["buckets"])
    assert np.array_equal(st.perm.cpu().numpy(), ref["perm"])
    err = np.abs(st.out.float().cpu().numpy() - ref["out"]).max()
    assert err <= out_tolerance(w.dtype), f"max-abs error {err}"
    assert lse_close(st.lse.cpu().numpy(), ref["lse"], w.dtype).all()
    return err


@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("chunk,L", [(64, 1024), (64, 1000), (128, 1024), (128, 1000)])
@pytest.mark.parametrize("after,across", [(1, False), (0, True), (1, True)])
def test_f32_lookahead_and_across(gpu, causal, chunk, L, after, across):
    """fp32 forward with one look-ahead chunk and/or attention across buckets,
    with chunks of 64 and 128 and a partial last chunk; mixture inputs, so
    buckets overflow the window."""
    w = small("mixture_bf16_L4096", B=1, H=2, L=L, n_rounds=3, n_buckets=16, chunk=chunk,
              causal=causal, dtype="f32")
    x = W.make_inputs(w)
    cfg = lsh.Config.of(w, chunks_after=after, attend_across=across)
    log("variant f32", causal, chunk, L, after, across)
    err = _forward(w, x["R"], cfg, after, across)
    print(f"f32 chunk={chunk} L={L} after={after} across={across} causal={causal}: err {err:.3e}")


@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("chunk,after,L", [(128, 0, 4096), (128, 0, 1000), (64, 1, 4096),
                                           (64, 1, 1000), (128, 1, 4096), (128, 1, 1000)])
def test_bf16_chunk128_and_lookahead(gpu, causal, chunk, after, L):
    """The bf16 matrix-core forward with chunks of 128 sorted slots (the
    paper's usual configuration, m = 2l/n_b, Sec. 5) and/or one look-ahead
    chunk, including a partial last chunk; 8 rounds of a 64-Gaussian mixture,
    so buckets are uneven and the window's masks span several 64-slot
    groups."""
    n_b = max(2, (2 * L // chunk) // 2 * 2)  # m = 2l/n_b, rounded to an even count
    w = small("long_bf16_L65536", H=2, L=L, n_components=64, n_buckets=n_b, chunk=chunk,
              causal=causal)
    x = W.make_inputs(w)
    cfg = lsh.Config.of(w, chunks_after=after)
    log("variant bf16", causal, chunk, after, L)
    err = _forward(w, x["R"], cfg, after)
    print(f"bf16 chunk={chunk} after={after} L={L} causal={causal}: err {err:.3e}")


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_r_per_head(gpu, dtype):
    """One R per head: each (batch, head) slice hashed with its head's R, bit
    for bit against the oracle's per-head hash, then the whole forward."""
    w = small("causal_bf16_L16384", B=2, H=3, L=2048, n_buckets=64, n_rounds=2, dtype=dtype)
    x = W.make_inputs(w)
    rng = np.random.default_rng(9)
    R = rng.standard_normal((w.H, w.n_rounds, w.d, w.n_buckets // 2)).astype(np.float32)
    cfg = lsh.Config.of(w, r_per_head=True)
    log("variant r_per_head", dtype)
    got = lsh.lsh_hash(cfg, to_device(x["q"], dtype), to_device(R, "f32")).cpu().numpy()
    want, near = oracle.lsh_hash(W.as_f64(x["q"], dtype), R.astype(np.float64))
    print(f"r_per_head {dtype}: near-tie row-rounds {int(near.sum())}")
    assert np.array_equal(got, want)
    # the heads really differ: the shared-R ids disagree somewhere
    shared, _ = oracle.lsh_hash(W.as_f64(x["q"], dtype), R[0].astype(np.float64))
    assert not np.array_equal(shared, want)
    _forward(w, R, cfg)
