"""Backward (dq, dv) of the GPU path against the fp64 oracle.

The GPU backward runs on the GPU forward's saved state (out, lse, buckets,
perm, undo, bucket_start); the oracle runs on its own forward.  Bucket ids are
bit-exact between the two, so both backward passes see the same problem.
Tolerance: 2e-2 max-abs (bf16 inputs, fp32 accumulation).
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2001_04451_amd import lsh
from paper_2001_04451_amd import workloads as W

from gpu_common import log, small, to_device

pytestmark = pytest.mark.gpu

TOL = 2e-2

CASES = {
    # the fwd+bwd workload reduced: causal, n_b = 512, 4 rounds
    "fwdbwd_small": small("fwdbwd_bf16_L32768", B=1, H=2, L=4096),
    # non-causal, clustered inputs, 2 rounds
    "mixture_small": small("mixture_bf16_L4096", B=1, H=2, L=2048, backward=True),
    # one round, causal, many tokens fall back to themselves
    "one_round": small("causal_bf16_L16384", B=1, H=1, L=1024, n_rounds=1, n_buckets=64,
                       backward=True),
    # eight rounds (four signature words), causal, clustered
    "eight_rounds": small("long_bf16_L65536", H=1, L=4096, n_buckets=256, backward=True),
    # an odd round count: a half-filled signature word, non-causal
    "three_rounds": small("mixture_bf16_L4096", B=1, H=1, L=2048, n_rounds=3, backward=True),
    # the most rounds the library takes (eight signature words), causal
    "sixteen_rounds": small("long_bf16_L65536", H=1, L=2048, n_buckets=256, n_rounds=16,
                            backward=True),
    # a partial last chunk (L mod 64 = 32), causal and not
    "partial_chunk_causal": small("fwdbwd_bf16_L32768", B=1, H=1, L=1056, n_buckets=64),
    "partial_chunk": small("mixture_bf16_L4096", B=1, H=1, L=1000, backward=True),
}


@pytest.fixture(scope="module")
def gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    lsh.lib()
    return torch.device("cuda:0")


def _run(w, slices=None):
    x = W.make_inputs(w, with_dout=True)
    cfg = lsh.Config.of(w)
    q, v, dout = (to_device(x[k], "bf16") for k in ("q", "v", "dout"))
    log("backward", w)
    st = lsh.lsh_attention_fwd(cfg, q, v, to_device(x["R"], "f32"))
    dq, dv = lsh.lsh_chunk_attn_bwd(cfg, q, v, st.out, dout, st.lse, st.buckets, st.perm,
                                    st.undo, st.bstart)
    torch.cuda.synchronize()
    dq, dv = dq.cpu().numpy(), dv.cpu().numpy()
    assert np.isfinite(dq).all() and np.isfinite(dv).all()
    R = x["R"].astype(np.float64)
    picks = slices or [(b, h) for b in range(w.B) for h in range(w.H)]
    # the chosen slices as one batch of one head each: the oracle runs them in parallel
    cat = lambda a: np.concatenate([a[b:b + 1, h:h + 1] for b, h in picks], axis=0)
    q64, v64, d64 = (W.as_f64(cat(x[k]), "bf16") for k in ("q", "v", "dout"))
    ref = oracle.lsh_attention_fwd(q64, v64, R, w.chunk, w.causal)
    assert np.array_equal(cat(st.buckets.cpu().numpy()), ref["buckets"])
    rdq, rdv = oracle.lsh_chunk_attn_bwd(q64, v64, ref["out"], d64, ref["lse"], ref["buckets"],
                                         ref["perm"], w.chunk, w.causal)
    eq = np.abs(cat(dq) - rdq).max()
    ev = np.abs(cat(dv) - rdv).max()
    print(f"{w.name} {len(picks)} slices: dq err {eq:.3e} (|dq| max {np.abs(rdq).max():.2f}), "
          f"dv err {ev:.3e} (|dv| max {np.abs(rdv).max():.2f})")
    return max(eq, ev)


@pytest.mark.parametrize("name", list(CASES))
def test_backward_small(gpu, name):
    assert _run(CASES[name]) <= TOL


def test_backward_full_size(gpu):
    """The fwd+bwd workload at its full size (B=8, H=8, L=32768, 4 rounds);
    the oracle recomputes eight whole (batch, head) slices, one per batch
    entry at spread heads."""
    w = W.WORKLOADS["fwdbwd_bf16_L32768"]
    assert _run(w, slices=[(b, (3 * b + 1) % w.H) for b in range(w.B)]) <= TOL


def test_backward_deterministic(gpu):
    """Two backward calls on the same forward state give bit-identical dq and
    dv: every sum has a fixed order (no atomics)."""
    w = CASES["fwdbwd_small"]
    x = W.make_inputs(w, with_dout=True)
    cfg = lsh.Config.of(w)
    q, v, dout = (to_device(x[k], "bf16") for k in ("q", "v", "dout"))
    log("backward-determinism", w)
    st = lsh.lsh_attention_fwd(cfg, q, v, to_device(x["R"], "f32"))
    dq1, dv1 = lsh.lsh_chunk_attn_bwd(cfg, q, v, st.out, dout, st.lse, st.buckets, st.perm,
                                      st.undo, st.bstart)
    dq2, dv2 = lsh.lsh_chunk_attn_bwd(cfg, q, v, st.out, dout, st.lse, st.buckets, st.perm,
                                      st.undo, st.bstart)
    torch.cuda.synchronize()
    assert torch.equal(dq1.view(torch.int32), dq2.view(torch.int32))
    assert torch.equal(dv1.view(torch.int32), dv2.view(torch.int32))
