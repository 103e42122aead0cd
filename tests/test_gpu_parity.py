"""GPU path (through the C ABI) against the fp64 oracle, stage by stage.

Every input is drawn by the seeded generators of paper_2001_04451_amd.workloads
or by the test itself; nothing the GPU writes is fed to the oracle.  Bucket
ids, permutations and bucket offsets must be bit-exact; floating-point
outputs must be within 1e-5 (fp32) or 2e-2 (bf16, fp32 accumulation) max-abs.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2001_04451_amd import lsh
from paper_2001_04451_amd import workloads as W

from gpu_common import log, lse_close, out_tolerance, rounds_f64, small, to_device, torch_dtype

pytestmark = pytest.mark.gpu

# Reduced copies of the five workloads: same n_b, n_r, dtype, causal flag and
# input distribution; sizes span several chunks, rows blocks and sort tiles.
SMALL = {
    "tiny_f32_L1024": small("tiny_f32_L1024"),
    "mixture_bf16_L4096": small("mixture_bf16_L4096", B=2, H=2),
    "causal_bf16_L16384": small("causal_bf16_L16384", B=1, H=2, L=4096),
    "long_bf16_L65536": small("long_bf16_L65536", H=1, L=8192),
    "fwdbwd_bf16_L32768": small("fwdbwd_bf16_L32768", B=1, H=2, L=4096),
}


def _inputs(w):
    x = W.make_inputs(w)
    q64, v64 = W.as_f64(x["q"], w.dtype), W.as_f64(x["v"], w.dtype)
    return x, q64, v64


@pytest.fixture(scope="module")
def gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    lsh.lib()
    return torch.device("cuda:0")


@pytest.mark.parametrize("name", list(SMALL))
def test_hash_bit_exact(gpu, name):
    w = SMALL[name]
    x, q64, _ = _inputs(w)
    want, near = oracle.lsh_hash(q64, x["R"].astype(np.float64))
    cfg = lsh.Config.of(w)
    log("hash", name, w)
    got = lsh.lsh_hash(cfg, to_device(x["q"], w.dtype), to_device(x["R"], "f32")).cpu().numpy()
    mism = got != want
    print(f"{name}: near-tie row-rounds {int(near.sum())}, mismatches {int(mism.sum())}"
          f" (all inside near ties: {bool((~mism | near).all())})")
    assert not (mism & ~near).any(), "bucket id differs outside the near-tie set"
    assert mism.sum() == 0


@pytest.mark.parametrize("n_buckets,L,n_rounds,B,H", [
    (2, 64, 1, 1, 1), (16, 1024, 1, 1, 1), (64, 4096, 2, 2, 3), (1024, 8192, 3, 1, 2),
    (1024, 4160, 2, 1, 1), (512, 12352, 4, 1, 1), (256, 64, 16, 2, 1),
    (1024, 65536, 2, 1, 1), (1024, 69632, 2, 1, 1),
    (14, 1001, 3, 1, 2), (1024, 4100, 2, 1, 1), (256, 37, 2, 2, 1)])
def test_sort_bit_exact(gpu, n_buckets, L, n_rounds, B, H):
    """Counting sort vs the oracle on test-drawn ids, including ragged tiles
    (L not a multiple of 4096), empty buckets and one-bucket segments.  The
    shapes with L = 65536 and 69632 have 16 tiles of 4096 positions, the
    most the scan holds in registers, and 17, which takes its general loop;
    L = 1001, 4100 and 37 are not multiples of 8 (the 16-bit id copy's
    element-wise path), and 14 buckets are not a multiple of four."""
    rng = np.random.Generator(np.random.PCG64(L + n_buckets))
    b = rng.integers(0, n_buckets, size=(B, H, L, n_rounds)).astype(np.int32)
    b[0, 0, :, 0] = n_buckets - 1  # one segment entirely in the last bucket
    if n_buckets >= 64:
        b[..., -1] = rng.integers(0, 3, size=(B, H, L))  # a segment with few buckets
    perm_want, undo_want = oracle.lsh_sort_permute(b)
    cfg = lsh.Config(B=B, H=H, L=L, n_buckets=n_buckets, n_rounds=n_rounds)
    log("sort", B, H, L, n_rounds, n_buckets)
    perm, undo, bstart = lsh.lsh_sort_permute(cfg, torch.from_numpy(b).cuda())
    assert np.array_equal(perm.cpu().numpy(), perm_want)
    assert np.array_equal(undo.cpu().numpy(), undo_want)
    # first sorted slot of every bucket, last entry L
    bs = bstart.cpu().numpy()
    for bb in range(B):
        for hh in range(H):
            for r in range(n_rounds):
                keys = b[bb, hh, :, r][perm_want[bb, hh, r]]
                want_bs = np.searchsorted(keys, np.arange(n_buckets + 1), side="left")
                assert np.array_equal(bs[bb, hh, r], want_bs)


@pytest.mark.parametrize("name", list(SMALL))
def test_chunk_attention_and_combine(gpu, name):
    """Attention and combine on oracle-drawn bucket ids (the oracle's own
    hash of the generator's q), sorted on the GPU."""
    w = SMALL[name]
    x, q64, v64 = _inputs(w)
    ref = oracle.lsh_attention_fwd(q64, v64, x["R"].astype(np.float64), w.chunk, w.causal)
    cfg = lsh.Config.of(w)
    q, v = to_device(x["q"], w.dtype), to_device(x["v"], w.dtype)
    buckets = torch.from_numpy(ref["buckets"]).cuda()
    log("attn", name, w)
    perm, undo, bstart = lsh.lsh_sort_permute(cfg, buckets)
    o_r, o_e, lse_r = lsh.lsh_chunk_attn_fwd(cfg, q, v, buckets, perm, bstart)
    out, lse = lsh.lsh_combine_rounds(cfg, o_r, o_e, lse_r, undo, torch_dtype(w.dtype))
    torch.cuda.synchronize()
    tol = out_tolerance(w.dtype)
    err_or = np.abs(rounds_f64(o_r, o_e) - ref["o_rounds"]).max()
    assert err_or <= tol, f"per-round output max-abs error {err_or}"
    assert lse_close(lse_r.cpu().numpy(), ref["lse_rounds"], w.dtype).all()
    got = out.float().cpu().numpy()
    err = np.abs(got - ref["out"]).max()
    print(f"{name}: out max-abs err {err:.3e} (tol {tol})")
    assert err <= tol
    assert lse_close(lse.cpu().numpy(), ref["lse"], w.dtype).all()


@pytest.mark.parametrize("name", list(SMALL))
def test_end_to_end_forward(gpu, name):
    """lsh_attention_fwd (all four stages chained in the library) vs the oracle."""
    w = SMALL[name]
    x, q64, v64 = _inputs(w)
    ref = oracle.lsh_attention_fwd(q64, v64, x["R"].astype(np.float64), w.chunk, w.causal)
    cfg = lsh.Config.of(w)
    log("forward", name, w)
    st = lsh.lsh_attention_fwd(cfg, to_device(x["q"], w.dtype), to_device(x["v"], w.dtype),
                               to_device(x["R"], "f32"))
    torch.cuda.synchronize()
    assert np.array_equal(st.buckets.cpu().numpy(), ref["buckets"])
    assert np.array_equal(st.perm.cpu().numpy(), ref["perm"])
    assert np.array_equal(st.undo.cpu().numpy(), ref["undo"])
    err = np.abs(st.out.float().cpu().numpy() - ref["out"]).max()
    print(f"{name}: end-to-end max-abs err {err:.3e}")
    assert err <= out_tolerance(w.dtype)
    assert lse_close(st.lse.cpu().numpy(), ref["lse"], w.dtype).all()


def test_forward_deterministic(gpu):
    w = SMALL["long_bf16_L65536"]
    x = W.make_inputs(w)
    cfg = lsh.Config.of(w)
    q, v, R = to_device(x["q"], w.dtype), to_device(x["v"], w.dtype), to_device(x["R"], "f32")
    log("determinism", w)
    a = lsh.lsh_attention_fwd(cfg, q, v, R)
    out_a = a.out.clone()
    b = lsh.lsh_attention_fwd(cfg, q, v, R)
    assert torch.equal(out_a.view(torch.int16), b.out.view(torch.int16))


def test_gather_rows(gpu):
    w = SMALL["mixture_bf16_L4096"]
    x = W.make_inputs(w)
    cfg = lsh.Config.of(w)
    q = to_device(x["q"], w.dtype)
    buckets = torch.from_numpy(oracle.lsh_hash(W.as_f64(x["q"], w.dtype), x["R"])[0]).cuda()
    log("gather", w)
    perm, _, _ = lsh.lsh_sort_permute(cfg, buckets)
    got = lsh.lsh_gather_rows(cfg, q, perm)
    p = perm.long()
    want = torch.stack([torch.stack([q[b, h][p[b, h, r]] for r in range(w.n_rounds)])
                        for b in range(w.B) for h in range(w.H)]).view(got.shape)
    assert torch.equal(got.view(torch.int16), want.view(torch.int16))


def test_invalid_arguments_on_gpu(gpu):
    cfg = lsh.Config(B=1, H=1, L=100, n_buckets=15, n_rounds=1)  # odd n_buckets
    q = torch.zeros((1, 1, 100, 64), device=gpu)
    R = torch.zeros((1, 64, 7), device=gpu)
    with pytest.raises(lsh.LshError) as e:
        lsh.lsh_hash(cfg, q, R)
    assert e.value.status == lsh.LSH_ERR_INVALID


@pytest.mark.parametrize("causal", [True, False])
@pytest.mark.parametrize("variant", ["large_norm", "duplicates_and_zeros", "large_values"])
def test_attention_edge_inputs(gpu, variant, causal):
    """Attention on edited inputs, with the oracle's bucket ids.

    large_norm: every fifth query scaled by 64, so its logit bound
    scale*log2(e)*|q| is far above the range the kernel covers without a
    running maximum; the waves holding such rows take the online-maximum path.
    duplicates_and_zeros: pairs of identical tokens (N_ij = n_r, the largest
    repeat count) and all-zero rows (zero norm, every logit zero).
    large_values: every value row times 2^17, so the per-round rows pass
    fp16's range and are stored with a nonzero exponent; the softmax weights
    do not change, so outputs and their errors scale by 2^17 and so does the
    tolerance."""
    w = small("mixture_bf16_L4096", B=1, H=2, L=2048, causal=causal)
    x = W.make_inputs(w)
    qf = W.bf16_bits_to_f32(x["q"])
    scale = 1.0
    if variant == "large_norm":
        qf[:, :, ::5, :] *= 64.0
    elif variant == "duplicates_and_zeros":
        qf[:, :, 1::4, :] = qf[:, :, 0::4, :]
        qf[:, :, 2::16, :] = 0.0
    else:
        scale = 2.0 ** 17
        x["v"] = W.f32_to_bf16_bits(W.bf16_bits_to_f32(x["v"]) * np.float32(scale))
    x["q"] = W.f32_to_bf16_bits(qf)
    q64, v64 = W.as_f64(x["q"], w.dtype), W.as_f64(x["v"], w.dtype)
    ref = oracle.lsh_attention_fwd(q64, v64, x["R"].astype(np.float64), w.chunk, w.causal)
    cfg = lsh.Config.of(w)
    q, v = to_device(x["q"], w.dtype), to_device(x["v"], w.dtype)
    buckets = torch.from_numpy(ref["buckets"]).cuda()
    log("attn-edge", variant, w)
    perm, undo, bstart = lsh.lsh_sort_permute(cfg, buckets)
    o_r, o_e, lse_r = lsh.lsh_chunk_attn_fwd(cfg, q, v, buckets, perm, bstart)
    out, lse = lsh.lsh_combine_rounds(cfg, o_r, o_e, lse_r, undo, torch.bfloat16)
    torch.cuda.synchronize()
    tol = out_tolerance(w.dtype) * scale
    if scale > 1.0:
        assert (o_e.cpu().numpy() > 0).any()  # the scaled form is exercised
    err_or = np.abs(rounds_f64(o_r, o_e) - ref["o_rounds"]).max()
    print(f"{variant} causal={causal}: per-round err {err_or:.3e} (tol {tol:.3g})")
    assert err_or <= tol
    assert lse_close(lse_r.cpu().numpy(), ref["lse_rounds"], w.dtype).all()
    got = out.float().cpu().numpy()
    err = np.abs(got - ref["out"]).max()
    print(f"{variant} causal={causal}: out max-abs err {err:.3e}")
    assert err <= tol
    assert lse_close(lse.cpu().numpy(), ref["lse"], w.dtype).all()


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_hash_exact_ties(gpu, dtype):
    """Exact ties in [xR; -xR]: a duplicated column, a negated column and
    all-zero queries.  The first index of [xR; -xR] must win, as in the
    oracle; every such row-round goes through the exact second pass."""
    w = small("mixture_bf16_L4096", B=1, H=2, L=2048, n_buckets=64, dtype=dtype)
    x = W.make_inputs(w)
    R = x["R"].copy()
    half = w.n_buckets // 2
    R[:, :, 9] = R[:, :, 5]      # x.R_9 == x.R_5: entry 5 beats entry 9
    R[:, :, 7] = -R[:, :, 3]     # x.R_7 == -x.R_3: entry 7 beats entry half+3
    q = x["q"].copy()
    q[:, :, ::37, :] = 0         # all projections zero: entry 0 wins
    q64 = W.as_f64(q, dtype)
    want, near = oracle.lsh_hash(q64, R.astype(np.float64))
    cfg = lsh.Config.of(w)
    log("hash-ties", dtype, w)
    got = lsh.lsh_hash(cfg, to_device(q, dtype), to_device(R, "f32")).cpu().numpy()
    print(f"{dtype}: near-tie row-rounds {int(near.sum())}, zero-row ids {np.unique(want[:, :, ::37])}, "
          f"ids 9 {(want == 9).sum()}, ids {half + 3}: {(want == half + 3).sum()}")
    assert (want[:, :, ::37] == 0).all()
    assert not (want == 9).any() and not (want == half + 3).any()
    assert np.array_equal(got, want)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("n_buckets", [2, 6, 66, 128, 200, 640, 1022])
def test_hash_bucket_counts(gpu, dtype, n_buckets):
    """Bucket counts the five workloads do not use: rounds of 1 to 511
    columns, so R's stages hold 1, 2, 4, 8 or 16 tiles and the last tile or
    stage of a round is partial.  Bit for bit against the oracle."""
    w = small("causal_bf16_L16384", B=1, H=2, L=1536, n_buckets=n_buckets, n_rounds=2, dtype=dtype)
    x, q64, _ = _inputs(w)
    want, near = oracle.lsh_hash(q64, x["R"].astype(np.float64))
    cfg = lsh.Config.of(w)
    log("hash-buckets", dtype, n_buckets)
    got = lsh.lsh_hash(cfg, to_device(x["q"], dtype), to_device(x["R"], "f32")).cpu().numpy()
    print(f"{dtype} n_b={n_buckets}: near-tie row-rounds {int(near.sum())}, mismatches {int((got != want).sum())}")
    assert np.array_equal(got, want)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_hash_extreme_scales(gpu, dtype):
    """Rows and rounds far from unit scale.  Each round's R is scaled by a
    power of two (2^-60, 1, 2^50 for bf16 input; 2^-30, 1, 2^30 for fp32);
    query rows are scaled by 2^k with k spread over [-100, 100] (bf16) or
    [-40, 40] (fp32), and for bf16 input some rows also hold a few values
    2^30 times larger than the rest (after the row's scaling the small ones
    fall below binary16's normal range) or lie in bf16's subnormal range.
    The argmax is scale invariant and the GPU's ids must equal the fp64
    oracle's everywhere."""
    w = small("causal_bf16_L16384", B=1, H=2, L=2048, n_buckets=256, n_rounds=3, dtype=dtype)
    x = W.make_inputs(w)
    R = x["R"].astype(np.float32).copy()
    q = W.as_f64(x["q"], dtype).astype(np.float32).reshape(-1, w.d)
    rng = np.random.default_rng(5150)
    kmax = 100 if dtype == "bf16" else 40
    rows = q.shape[0]
    k = rng.integers(-kmax, kmax + 1, rows)
    q = q * np.ldexp(1.0, k)[:, None].astype(np.float32)
    if dtype == "bf16":
        R[0] *= np.float32(2.0 ** -60)
        R[1] *= np.float32(2.0 ** 50)
        wide = np.arange(rows) % 4 == 1  # a few large values beside small ones
        q[wide] *= np.float32(2.0 ** -40)  # stays inside fp32's range
        q[wide, :4] *= np.float32(2.0 ** 30)
        sub = np.arange(rows) % 4 == 2   # bf16 subnormals (below 2^-126)
        q[sub] = (W.as_f64(x["q"], dtype).reshape(-1, w.d)[sub] * 2.0 ** -130).astype(np.float32)
        qin = W.f32_to_bf16_bits(q).reshape(x["q"].shape)
    else:
        R[0] *= np.float32(2.0 ** -30)
        R[1] *= np.float32(2.0 ** 30)
        qin = q.reshape(x["q"].shape)
    q64 = W.as_f64(qin, dtype)
    assert np.isfinite(q64).all() and (np.abs(q64).max(axis=-1) > 0).all()
    want, near = oracle.lsh_hash(q64, R.astype(np.float64))
    cfg = lsh.Config.of(w)
    log("hash-scales", dtype)
    got = lsh.lsh_hash(cfg, to_device(qin, dtype), to_device(R, "f32")).cpu().numpy()
    print(f"{dtype}: near-tie row-rounds {int(near.sum())}, mismatches {int((got != want).sum())}")
    assert np.array_equal(got, want)


def _rounds_input(o: np.ndarray, dtype: str, rng):
    """Per-round rows in the format lsh_combine_rounds takes for `dtype`, and
    their exact float64 values.  For bf16 calls: fp16 rows with a per-row
    exponent; with `rng`, every 97th row is scaled up by 2^20 and stored with
    exponent 20 (the form the attention writes for rows past fp16's range)."""
    if dtype == "f32":
        return torch.from_numpy(o).cuda(), None, o.astype(np.float64)
    e = np.zeros(o.shape[:-1], np.uint8)
    if rng is not None:
        e.reshape(-1)[::97] = 20
    h = o.astype(np.float16)
    o64 = np.ldexp(h.astype(np.float64), e.astype(np.int32)[..., None])
    return torch.from_numpy(h).cuda(), torch.from_numpy(e).cuda(), o64


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("n_rounds", [3, 6, 9, 16])
def test_combine_round_counts(gpu, dtype, n_rounds):
    """The combine for round counts the five workloads do not use: counts that
    are not a power of two (rounds past n_r padded inside the kernel) and
    counts above 8 (two rounds per lane).  Per-round rows, log-partitions and
    the inverse permutations are drawn here."""
    B, H, L, d = 1, 2, 1024, 64
    rng = np.random.default_rng(1000 + n_rounds)
    o = rng.standard_normal((B, H, n_rounds, L, d)).astype(np.float32)
    lse_r = (5.0 * rng.standard_normal((B, H, n_rounds, L))).astype(np.float32)
    undo = np.stack([np.stack([np.argsort(rng.permutation(L)) for _ in range(n_rounds)])
                     for _ in range(B * H)]).reshape(B, H, n_rounds, L).astype(np.int32)
    o_r, o_e, o64 = _rounds_input(o, dtype, rng)
    ref_out, ref_lse = oracle.lsh_combine_rounds(o64, lse_r.astype(np.float64), undo)
    cfg = lsh.Config(B=B, H=H, L=L, n_buckets=64, n_rounds=n_rounds)
    tdt = torch_dtype(dtype)
    log("combine", dtype, n_rounds)
    out, lse = lsh.lsh_combine_rounds(cfg, o_r, o_e, torch.from_numpy(lse_r).cuda(),
                                      torch.from_numpy(undo).cuda(), tdt)
    torch.cuda.synchronize()
    got = out.float().cpu().numpy()
    if o_e is None:
        big = np.zeros(ref_lse.shape, bool)
    else:  # tokens with a scaled row in some round: outputs near 2^20
        e_tok = np.take_along_axis(o_e.cpu().numpy(), undo.astype(np.int64), axis=3)
        big = (e_tok > 0).any(axis=2)
    err = np.abs(got - ref_out)[~big].max()
    assert err <= out_tolerance(dtype), f"combine max-abs error {err}"
    if big.any():
        # outputs of magnitude ~2^20: one bf16 rounding (2^-8 relative) plus
        # fp32 accumulation, relative to the row's scale
        rel = np.abs(got - ref_out)[big] / (2.0 ** -8 * np.abs(ref_out)[big] + 2.0 ** -20 * 2.0 ** 20)
        assert rel.max() <= 1.0, f"scaled rows: error {rel.max()} of the bound"
    assert lse_close(lse.cpu().numpy(), ref_lse, dtype).all()


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_combine_lone_token_weights(gpu, dtype):
    """Tokens alone in their buckets in every round: each z_r sits near
    -self_mask (where one fp32 spacing is 2^-7), and mixed rows put such a
    round beside ordinary ones.  The weights must not inherit the rounding of
    z at that magnitude: equal z_r give the mean of the rows to fp32
    accuracy."""
    B, H, L, d, n_rounds = 1, 1, 512, 64, 3
    rng = np.random.default_rng(77)
    o = rng.standard_normal((B, H, n_rounds, L, d)).astype(np.float32)
    o_r, o_e, o64 = _rounds_input(o, dtype, None)
    base = (-1e5 + 2.0 + rng.standard_normal((B, H, 1, L))).astype(np.float32)
    lse_r = np.repeat(base, n_rounds, axis=2)
    # every fourth token: round 1 has other targets (an ordinary z_r)
    lse_r[:, :, 1, ::4] = rng.standard_normal(L // 4).astype(np.float32)
    undo = np.stack([np.argsort(rng.permutation(L)) for _ in range(n_rounds)]).reshape(
        B, H, n_rounds, L).astype(np.int32)
    ref_out, ref_lse = oracle.lsh_combine_rounds(o64, lse_r.astype(np.float64), undo)
    cfg = lsh.Config(B=B, H=H, L=L, n_buckets=64, n_rounds=n_rounds)
    tdt = torch_dtype(dtype)
    log("combine-lone", dtype)
    out, lse = lsh.lsh_combine_rounds(cfg, o_r, o_e, torch.from_numpy(lse_r).cuda(),
                                      torch.from_numpy(undo).cuda(), tdt)
    torch.cuda.synchronize()
    diff = np.abs(out.float().cpu().numpy() - ref_out)
    # bf16 output: the weighted mean to fp32 accuracy, then one rounding to
    # nearest (half an ulp of an 8-bit significand: at most 2^-8 relative)
    bound = 1e-5 if dtype == "f32" else np.minimum(2.0 ** -8 * np.abs(ref_out) + 1e-6, 2e-2)
    assert (diff <= bound).all(), f"combine max-abs error {diff.max()}"
    assert lse_close(lse.cpu().numpy(), ref_lse, dtype).all()


def test_hash_listed_pass_many_open_rows(gpu):
    """Round 0's queries are built as near-ties between two columns of R, so
    the hi-plane screen leaves nearly every row of that round open: each
    segment of the list then holds more rows than its workgroups take in one
    pass and they loop over its chunks.  Round 1 is ordinary.  262144 rows;
    4096 of them, drawn at random, are checked against the oracle bit for
    bit."""
    B, H, L, n_b, n_r, d = 1, 4, 65536, 1024, 2, 64
    half = n_b // 2
    rng = np.random.default_rng(4242)
    R = rng.standard_normal((n_r, d, half)).astype(np.float32)
    rows = B * H * L
    a = rng.integers(0, half, rows)
    b = (a + 1 + rng.integers(0, half - 1, rows)) % half
    Ra, Rb = R[0][:, a].T.astype(np.float64), R[0][:, b].T.astype(np.float64)  # [rows, d]
    gaa, gbb, gab = (Ra * Ra).sum(1), (Rb * Rb).sum(1), (Ra * Rb).sum(1)
    # q = alpha R_a + beta R_b with q.R_a = 1 and q.R_b = 1 - 1e-4
    det = gaa * gbb - gab * gab
    ta, tb = np.ones(rows), np.full(rows, 1 - 1e-4)
    alpha, beta = (gbb * ta - gab * tb) / det, (gaa * tb - gab * ta) / det
    q32 = (alpha[:, None] * Ra + beta[:, None] * Rb).astype(np.float32)
    q_bf = torch.from_numpy(q32).to(torch.bfloat16).reshape(B, H, L, d)
    cfg = lsh.Config(B=B, H=H, L=L, n_buckets=n_b, n_rounds=n_r)
    log("hash-listed-loop", rows)
    got = lsh.lsh_hash(cfg, q_bf.cuda(), torch.from_numpy(R).cuda()).cpu().numpy().reshape(rows, n_r)
    pick = np.sort(rng.choice(rows, 4096, replace=False))
    q64 = q_bf.float().numpy().astype(np.float64).reshape(rows, d)[pick].reshape(1, 1, -1, d)
    want, near = oracle.lsh_hash(q64, R.astype(np.float64))
    want = want.reshape(-1, n_r)
    top2 = np.isin(want[:, 0] % half, np.stack([a[pick], b[pick]], 1)).mean()
    print(f"round 0 winner among the two built columns: {top2:.3f}; near-ties {int(near.sum())}")
    assert top2 > 0.9  # the construction does what it is meant to
    assert np.array_equal(got[pick], want)


@pytest.mark.parametrize("causal", [True, False])
@pytest.mark.parametrize("n_rounds", [3, 6, 11, 16])
def test_forward_round_counts(gpu, n_rounds, causal):
    """The whole forward for round counts the five workloads do not use: an
    odd count (a half-filled signature word), and 6, 11 and 16 rounds (3, 6
    and 8 signature words, two rounds per lane in the combine above 8).
    Mixture inputs, so buckets are uneven and N_ij often exceeds 1."""
    w = small("mixture_bf16_L4096", B=1, H=2, L=2048, n_rounds=n_rounds, causal=causal)
    x, q64, v64 = _inputs(w)
    ref = oracle.lsh_attention_fwd(q64, v64, x["R"].astype(np.float64), w.chunk, w.causal)
    cfg = lsh.Config.of(w)
    log("forward-rounds", n_rounds, causal, w)
    st = lsh.lsh_attention_fwd(cfg, to_device(x["q"], w.dtype), to_device(x["v"], w.dtype),
                               to_device(x["R"], "f32"))
    torch.cuda.synchronize()
    assert np.array_equal(st.buckets.cpu().numpy(), ref["buckets"])
    assert np.array_equal(st.perm.cpu().numpy(), ref["perm"])
    err = np.abs(st.out.float().cpu().numpy() - ref["out"]).max()
    print(f"n_r={n_rounds} causal={causal}: max-abs err {err:.3e}")
    assert err <= out_tolerance(w.dtype)
    assert lse_close(st.lse.cpu().numpy(), ref["lse"], w.dtype).all()



@pytest.mark.parametrize("dtype,causal,L", [("bf16", True, 4000), ("bf16", False, 4000),
                                            ("bf16", True, 100), ("bf16", False, 130),
                                            ("f32", True, 1000), ("f32", False, 70)])
def test_forward_partial_last_chunk(gpu, dtype, causal, L):
    """L not a multiple of the chunk: the last chunk holds the L mod 64
    remaining slots (no key or query past L).  Whole forward against the
    oracle, which pins this reading against the dense windowed form."""
    w = small("mixture_bf16_L4096", B=1, H=2, L=L, n_rounds=3, causal=causal, dtype=dtype)
    x, q64, v64 = _inputs(w)
    ref = oracle.lsh_attention_fwd(q64, v64, x["R"].astype(np.float64), w.chunk, w.causal)
    cfg = lsh.Config.of(w)
    log("forward-partial-chunk", dtype, causal, L)
    st = lsh.lsh_attention_fwd(cfg, to_device(x["q"], w.dtype), to_device(x["v"], w.dtype),
                               to_device(x["R"], "f32"))
    torch.cuda.synchronize()
    assert np.array_equal(st.buckets.cpu().numpy(), ref["buckets"])
    assert np.array_equal(st.perm.cpu().numpy(), ref["perm"])
    err = np.abs(st.out.float().cpu().numpy() - ref["out"]).max()
    print(f"{dtype} causal={causal} L={L}: max-abs err {err:.3e}")
    assert err <= out_tolerance(w.dtype)
    assert lse_close(st.lse.cpu().numpy(), ref["lse"], w.dtype).all()


@pytest.mark.parametrize("causal,L", [(True, 1024), (False, 1024), (True, 1000), (False, 333)])
def test_forward_chunk_128(gpu, causal, L):
    """Chunks of 128 sorted slots (the paper's usual configuration, Sec. 5,
    with m = 2l/n_b: 16 buckets at L = 1024) on the fp32 path: whole forward
    against the oracle, including a partial last chunk."""
    w = small("tiny_f32_L1024", L=L, chunk=128, n_buckets=16, n_rounds=3, causal=causal)
    x, q64, v64 = _inputs(w)
    ref = oracle.lsh_attention_fwd(q64, v64, x["R"].astype(np.float64), w.chunk, w.causal)
    cfg = lsh.Config.of(w)
    log("forward-chunk-128", causal, L)
    st = lsh.lsh_attention_fwd(cfg, to_device(x["q"], "f32"), to_device(x["v"], "f32"),
                               to_device(x["R"], "f32"))
    torch.cuda.synchronize()
    assert np.array_equal(st.buckets.cpu().numpy(), ref["buckets"])
    assert np.array_equal(st.perm.cpu().numpy(), ref["perm"])
    err = np.abs(st.out.float().cpu().numpy() - ref["out"]).max()
    print(f"chunk 128 causal={causal} L={L}: max-abs err {err:.3e}")
    assert err <= out_tolerance("f32")
    assert lse_close(st.lse.cpu().numpy(), ref["lse"], "f32").all()

