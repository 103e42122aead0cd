"""GPU parity of the dense (full shared-QK) attention baseline against the
fp64 oracle: whole outputs at sizes the oracle finishes in seconds (several
key blocks and query workgroups, ragged tails, one-token sequences, the
online-maximum path), and sampled rows at the sizes the speed sweep times."""
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


def _bf16_bits_scaled(bits: np.ndarray, factor_log2: int) -> np.ndarray:
    """Multiply bf16 values (given as bit patterns) by 2^factor_log2 exactly."""
    t = torch.from_numpy(np.ascontiguousarray(bits)).view(torch.bfloat16) * (2.0 ** factor_log2)
    return t.view(torch.int16).numpy().view(bits.dtype)


def _run(B, H, L, causal, seed=1, big_rows=None):
    w = small("mixture_bf16_L4096", B=B, H=H, L=L, causal=causal, seed=seed)
    x = W.make_inputs(w)
    q = x["q"]
    if big_rows is not None:
        # logit bounds above the no-maximum range: these rows scaled by 64
        q = q.copy()
        q[..., big_rows, :] = _bf16_bits_scaled(q[..., big_rows, :], 6)
    cfg = lsh.Config(B=B, H=H, L=L, n_buckets=2, n_rounds=1, causal=causal)
    log("dense", B, H, L, causal, "big" if big_rows is not None else "")
    out, lse = lsh.lsh_dense_attn_fwd(cfg, to_device(q, "bf16"), to_device(x["v"], "bf16"))
    torch.cuda.synchronize()
    return q, x["v"], out.float().cpu().numpy(), lse.cpu().numpy()


@pytest.mark.parametrize("causal", [True, False])
@pytest.mark.parametrize("B,H,L", [(1, 2, 1000), (2, 1, 1024), (1, 1, 64), (1, 1, 130),
                                   (1, 1, 1), (1, 3, 200)])
def test_dense_matches_oracle(gpu, B, H, L, causal):
    q, v, out, lse = _run(B, H, L, causal)
    ref_out, ref_lse = oracle.dense_attn_fwd(W.as_f64(q, "bf16"), W.as_f64(v, "bf16"), causal)
    err = np.abs(out - ref_out).max()
    print(f"dense B={B} H={H} L={L} causal={causal}: max-abs err {err:.3e}")
    assert err <= out_tolerance("bf16")
    assert lse_close(lse, ref_lse, "bf16").all()


@pytest.mark.parametrize("causal", [True, False])
def test_dense_online_maximum(gpu, causal):
    """Queries whose logit bound exceeds the no-maximum range take the online
    maximum; every other wave keeps the fixed-bound softmax."""
    L = 700
    big = np.arange(0, L, 3)
    q, v, out, lse = _run(1, 2, L, causal, seed=3, big_rows=big)
    ref_out, ref_lse = oracle.dense_attn_fwd(W.as_f64(q, "bf16"), W.as_f64(v, "bf16"), causal)
    err = np.abs(out - ref_out).max()
    print(f"dense online-max causal={causal}: max-abs err {err:.3e}")
    assert err <= out_tolerance("bf16")
    assert lse_close(lse, ref_lse, "bf16").all()


@pytest.fixture(scope="module")
def headline_tokens():
    """The 64K-token, 16-head mixture inputs of the LSH benchmark, drawn once."""
    x = W.make_inputs(W.WORKLOADS["long_bf16_L65536"])
    return x["q"], x["v"]


# the configurations the speed sweep times at its ends (1M tokens x heads):
# the same tokens, as one 64K sequence or as 64 sequences of 1K
@pytest.mark.parametrize("B,H,L", [(1, 16, 65536), (64, 16, 1024)])
def test_dense_full_size_sampled_rows(gpu, headline_tokens, B, H, L):
    q, v = (np.ascontiguousarray(t.reshape(H, B, L, 64).transpose(1, 0, 2, 3))
            for t in headline_tokens)
    cfg = lsh.Config(B=B, H=H, L=L, n_buckets=2, n_rounds=1, causal=True)
    log("dense full size", B, H, L)
    out, lse = lsh.lsh_dense_attn_fwd(cfg, to_device(q, "bf16"), to_device(v, "bf16"))
    torch.cuda.synchronize()
    out, lse = out.float().cpu().numpy(), lse.cpu().numpy()
    rng = np.random.default_rng(L)
    n = B * H * L
    rows = np.unique(np.concatenate([
        [0, 1, 63, 64, 127, 128, L - 1, n - 1, n - L],   # block and sequence edges
        rng.integers(0, n, 48)]))
    ref_out, ref_lse = oracle.dense_attn_fwd(W.as_f64(q, "bf16"), W.as_f64(v, "bf16"), True,
                                             rows=rows)
    got = out.reshape(n, -1)[rows]
    err = np.abs(got - ref_out).max()
    print(f"dense full size B={B} H={H} L={L}: {len(rows)} rows, max-abs err {err:.3e}")
    assert err <= out_tolerance("bf16")
    assert lse_close(lse.reshape(-1)[rows], ref_lse, "bf16").all()
    assert np.isfinite(out).all()
