"""The five workloads at their full sizes, in the launch configuration the
benchmark times.  The GPU runs the whole batch; the oracle recomputes whole
(batch, head) slices of it (every slice is an independent problem), and the
rest of the batch is checked through properties that hold at any size."""
import numpy as np
import pytest
import torch

import oracle
from paper_2001_04451_amd import lsh
from paper_2001_04451_amd import workloads as W

from gpu_common import log, lse_close, out_tolerance, to_device

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    lsh.lib()
    return torch.device("cuda:0")


def _sorted_property(buckets: np.ndarray, perm: np.ndarray, undo: np.ndarray) -> None:
    """perm is a permutation ordering (bucket, position) strictly; undo inverts it."""
    B, H, nr, L = perm.shape
    for b in range(B):
        for h in range(H):
            for r in range(nr):
                p = perm[b, h, r].astype(np.int64)
                key = buckets[b, h, :, r].astype(np.int64)[p] * L + p
                assert (np.diff(key) > 0).all()
                assert np.array_equal(np.sort(p), np.arange(L))
                assert np.array_equal(undo[b, h, r][p], np.arange(L))


def _slices(x: dict, picks, key: str) -> np.ndarray:
    """The chosen (batch, head) slices of an input, stacked as a batch of one
    head each (every slice is an independent problem)."""
    return np.concatenate([x[key][b:b + 1, h:h + 1] for b, h in picks], axis=0)


def full_picks(w: W.Workload):
    """Every (batch, head) slice when there are at most 32; otherwise one per
    batch entry, at spread heads."""
    if w.B * w.H <= 32:
        return [(b, h) for b in range(w.B) for h in range(w.H)]
    return [(b, (3 * b + 1) % w.H) for b in range(w.B)]


@pytest.mark.parametrize("name", list(W.WORKLOADS))
def test_full_forward(gpu, name):
    w = W.WORKLOADS[name]
    x = W.make_inputs(w, with_dout=False)
    cfg = lsh.Config.of(w)
    log("full forward", name)
    st = lsh.lsh_attention_fwd(cfg, to_device(x["q"], w.dtype), to_device(x["v"], w.dtype),
                               to_device(x["R"], "f32"))
    torch.cuda.synchronize()
    buckets = st.buckets.cpu().numpy()
    perm, undo = st.perm.cpu().numpy(), st.undo.cpu().numpy()
    out = st.out.float().cpu().numpy()
    lse = st.lse.cpu().numpy()
    assert np.isfinite(out).all() and np.isfinite(lse).all()
    assert buckets.min() >= 0 and buckets.max() < w.n_buckets
    _sorted_property(buckets, perm, undo)
    R = x["R"].astype(np.float64)

    # bucket ids of rows sampled across every slice, against the oracle's hash
    rng = np.random.default_rng(11)
    n_sample = min(w.rows, 65536)
    flat = np.sort(rng.choice(w.rows, n_sample, replace=False))
    q_rows = x["q"].reshape(w.rows, w.d)[flat].reshape(1, 1, n_sample, w.d)
    want, near = oracle.lsh_hash(W.as_f64(q_rows, w.dtype), R)
    got = buckets.reshape(w.rows, w.n_rounds)[flat]
    mism = got != want.reshape(n_sample, w.n_rounds)
    print(f"{name} sampled rows {n_sample} of {w.rows}: near-tie row-rounds {int(near.sum())}, "
          f"bucket mismatches {int(mism.sum())}")
    assert mism.sum() == 0

    # whole slices through the oracle (all of them, or one per batch entry)
    picks = full_picks(w)
    q64 = W.as_f64(_slices(x, picks, "q"), w.dtype)
    v64 = W.as_f64(_slices(x, picks, "v"), w.dtype)
    ref = oracle.lsh_attention_fwd(q64, v64, R, w.chunk, w.causal)
    sel = lambda a: np.concatenate([a[b:b + 1, h:h + 1] for b, h in picks], axis=0)
    mism = sel(buckets) != ref["buckets"]
    print(f"{name}: {len(picks)} of {w.B * w.H} slices, near-tie row-rounds "
          f"{int(ref['near_tie'].sum())}, bucket mismatches {int(mism.sum())}")
    assert not (mism & ~ref["near_tie"]).any()
    assert mism.sum() == 0
    assert np.array_equal(sel(perm), ref["perm"])
    err = np.abs(sel(out) - ref["out"]).max()
    print(f"{name}: out max-abs err {err:.3e} over {len(picks)} slices")
    assert err <= out_tolerance(w.dtype)
    assert lse_close(sel(lse), ref["lse"], w.dtype).all()
