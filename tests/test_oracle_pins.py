"""Pins of the CPU oracle to what the paper and the mathematics fix.

None of these tests reuses the oracle's code: each expected value comes from
an independent NumPy/PyTorch formulation, a closed form, a brute-force
search or a hand-derived fixture.  Citations name the passage of the
Reformer paper (arXiv:2001.04451) each check follows.
"""
import json
import os

import numpy as np
import pytest
import torch

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# --------------------------------------------------------------------------
# independent references
# --------------------------------------------------------------------------
def _rng(seed):
    return np.random.Generator(np.random.PCG64(seed))


def _keys(q):
    n = np.linalg.norm(q, axis=-1, keepdims=True)
    return np.where(n > 0, q / np.where(n > 0, n, 1.0), 0.0)


def window_masks(buckets, chunk, after=0):
    """Per round, the [L, L] window membership of App. A's P~^(r) read from
    lexsort slots without any chunk loop: key j is in query i's window when
    floor(s_j/m) lies in floor(s_i/m) - 1 .. floor(s_i/m) + after."""
    L, n_r = buckets.shape
    pos = np.arange(L)
    masks = []
    for r in range(n_r):
        order = np.lexsort((pos, buckets[:, r]))
        slot = np.empty(L, np.int64)
        slot[order] = pos
        ci = slot // chunk
        masks.append((ci[None, :] >= ci[:, None] - 1) & (ci[None, :] <= ci[:, None] + after))
    return masks


def dense_logits(q, buckets, chunk, causal, scale, self_mask=1e5, after=0, across=False):
    """Logits a^(r)_ij of every (round, key) entry of every query, as dense
    [n_r, L, L] arrays with -inf where j is no target (App. A, m^(r)_ij).
    Across buckets the target set of a round is its window, and N_ij counts
    window memberships instead of shared buckets."""
    L, _ = q.shape
    n_r = buckets.shape[1]
    k = _keys(q)
    pos = np.arange(L)
    win = window_masks(buckets, chunk, after)
    if across:
        N = sum(w.astype(np.int64) for w in win)
    else:
        N = (buckets[:, None, :] == buckets[None, :, :]).sum(-1)
    with np.errstate(divide="ignore"):
        logN = np.log(N.astype(np.float64))
    M = np.where(np.eye(L, dtype=bool), self_mask, logN)
    out = np.empty((n_r, L, L))
    for r in range(n_r):
        ok = win[r].copy()
        if not across:
            ok &= buckets[:, r][:, None] == buckets[:, r][None, :]
        if causal:
            ok &= pos[None, :] <= pos[:, None]
        out[r] = np.where(ok, scale * (q @ k.T) - M, -np.inf)
    return out


def dense_output(q, v, buckets, chunk, causal, scale, self_mask=1e5, after=0, across=False):
    """The combined output as one softmax over every (round, key) entry."""
    a = dense_logits(q, buckets, chunk, causal, scale, self_mask, after, across)
    L = q.shape[0]
    flat = np.transpose(a, (1, 0, 2)).reshape(L, -1)  # [L, n_r * L]
    amax = flat.max(1, keepdims=True)
    w = np.exp(flat - amax)
    z = amax[:, 0] + np.log(w.sum(1))
    w /= w.sum(1, keepdims=True)
    vv = np.tile(v, (a.shape[0], 1))
    return w @ vv, z


def run_oracle(q, v, buckets, chunk, causal, scale=None, self_mask=1e5, after=0, across=False):
    """Oracle forward on one (b, h) slice with given bucket ids."""
    L, d = q.shape
    b4 = buckets.reshape(1, 1, L, -1)
    perm, undo = oracle.lsh_sort_permute(b4)
    o_r, lse_r = oracle.lsh_chunk_attn_fwd(q.reshape(1, 1, L, d), v.reshape(1, 1, L, d), b4,
                                           perm, chunk, causal, scale, self_mask, after, across)
    out, lse = oracle.lsh_combine_rounds(o_r, lse_r, undo)
    return out[0, 0], lse[0, 0], dict(perm=perm, undo=undo, o_r=o_r, lse_r=lse_r)


# --------------------------------------------------------------------------
# hand-derived worked example (tests/golden/worked_example_L6.json)
# --------------------------------------------------------------------------
def test_worked_example(oracle_lib):
    ex = json.load(open(os.path.join(GOLDEN, "worked_example_L6.json")))
    q = np.array(ex["q"], np.float64)
    v = np.array(ex["v"], np.float64)
    R = np.array(ex["R"], np.float64)
    L, d = q.shape
    buckets, _ = oracle.lsh_hash(q.reshape(1, 1, L, d), R)
    assert buckets[0, 0, :, 0].tolist() == ex["buckets"]
    perm, undo = oracle.lsh_sort_permute(buckets)
    assert perm[0, 0, 0].tolist() == ex["perm"]
    assert undo[0, 0, 0].tolist() == ex["undo"]
    scale = 1.0 / np.sqrt(d)
    k = _keys(q)
    for causal, key in ((False, "targets_noncausal"), (True, "targets_causal")):
        out, lse, _ = run_oracle(q, v, buckets[0, 0], ex["chunk"], causal)
        for i, T in enumerate(ex[key]):
            if T:
                a = np.array([scale * q[i] @ k[j] for j in T])
                w = np.exp(a - a.max())
                w /= w.sum()
                want = sum(wj * v[j] for wj, j in zip(w, T))
                assert np.allclose(out[i], want, atol=1e-14, rtol=0)
                assert abs(lse[i] - (a.max() + np.log(np.exp(a - a.max()).sum()))) < 1e-12
            else:
                # only target left is the token itself, with mask 1e5 (App. A)
                assert np.array_equal(out[i], v[i])
                assert abs(lse[i] - (scale * np.linalg.norm(q[i]) - 1e5)) < 1e-9


# --------------------------------------------------------------------------
# P1: one bucket, one chunk == dense shared-QK attention with self masked
# --------------------------------------------------------------------------
@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("L,d", [(64, 8), (128, 64), (256, 16)])
def test_one_bucket_is_dense_attention(oracle_lib, causal, L, d):
    """eq. attn with K = Q/|Q| (Sec. 2, shared-QK) and the self-exclusion of
    Sec. 2 'Causal masking for shared-QK attention'."""
    rng = _rng(L + d + causal)
    q = rng.standard_normal((L, d))
    v = rng.standard_normal((L, d))
    scale = 1.0 / np.sqrt(d)
    out, lse, _ = run_oracle(q, v, np.zeros((L, 1), np.int32), chunk=L, causal=causal)
    k = q / np.linalg.norm(q, axis=1, keepdims=True)
    s = scale * q @ k.T
    allowed = ~np.eye(L, dtype=bool)
    if causal:
        allowed &= np.tril(np.ones((L, L), bool))
    s = np.where(allowed, s, -np.inf)
    rows = allowed.any(1)
    sm = np.exp(s[rows] - s[rows].max(1, keepdims=True))
    sm /= sm.sum(1, keepdims=True)
    np.testing.assert_allclose(out[rows], sm @ v, atol=1e-12, rtol=0)
    if causal:
        # the first token has no earlier target and attends to itself
        assert not rows[0] and rows[1:].all()
        assert np.array_equal(out[0], v[0])
    else:
        assert rows.all()


# --------------------------------------------------------------------------
# P2 / P9: the hash against brute force, tie rule, invariances
# --------------------------------------------------------------------------
@pytest.mark.parametrize("n_buckets,n_rounds,d", [(2, 3, 8), (16, 1, 64), (64, 2, 64), (1024, 2, 64)])
def test_hash_brute_force(oracle_lib, n_buckets, n_rounds, d):
    """h(x) = argmax([xR; -xR]) (Sec. 2, 'Locality sensitive hashing')."""
    rng = _rng(n_buckets * 7 + n_rounds)
    L = 512
    q = rng.standard_normal((2, 1, L, d))
    R = rng.standard_normal((n_rounds, d, n_buckets // 2))
    buckets, near = oracle.lsh_hash(q, R)
    for r in range(n_rounds):
        p = q @ R[r]
        vals = np.concatenate([p, -p], axis=-1)
        want = np.argmax(vals, axis=-1)
        top2 = np.sort(vals, axis=-1)[..., -2:]
        want_near = (top2[..., 1] - top2[..., 0]) < 1e-6 * np.abs(top2[..., 1])
        assert np.array_equal(near[..., r], want_near)
        ok = ~want_near
        assert np.array_equal(buckets[..., r][ok], want[ok])


def test_hash_tie_rule(oracle_lib):
    """Exact ties go to the first index of [xR; -xR]: the + half before the -
    half, lower column first (reading of Sec. 2's argmax)."""
    d, half = 4, 4
    x = np.zeros((1, 1, 3, d))
    x[..., 0] = 1.0
    R = np.zeros((1, d, half))
    # row-independent R; check three tie layouts with separate rounds
    Rs = []
    R1 = R.copy(); R1[0, 0, 1] = 2.0; R1[0, 0, 3] = 2.0       # + tie at columns 1 and 3
    R2 = R.copy(); R2[0, 0, 2] = 2.0; R2[0, 0, 0] = -2.0      # +col 2 ties -col 0
    R3 = R.copy(); R3[0, 0, 1] = -2.0; R3[0, 0, 3] = -2.0     # - tie at columns 1 and 3
    Rs = np.concatenate([R1, R2, R3], axis=0)
    buckets, near = oracle.lsh_hash(x, Rs)
    assert buckets[0, 0, 0].tolist() == [1, 2, half + 1]
    assert near.all()


def test_hash_invariances(oracle_lib):
    rng = _rng(11)
    q = rng.standard_normal((1, 2, 300, 64))
    R = rng.standard_normal((3, 64, 128))
    b0, n0 = oracle.lsh_hash(q, R)
    for k in (-3, 5, 20):
        bk, nk = oracle.lsh_hash(q * 2.0 ** k, R)
        assert np.array_equal(b0, bk) and np.array_equal(n0, nk)
    # two buckets: h(x) = 0 iff x.R >= 0
    R2 = rng.standard_normal((1, 64, 1))
    b2, _ = oracle.lsh_hash(q, R2)
    assert np.array_equal(b2[..., 0], np.where((q @ R2[0])[..., 0] >= 0, 0, 1))


def test_hash_zero_vector(oracle_lib):
    q = np.zeros((1, 1, 2, 8))
    R = _rng(3).standard_normal((2, 8, 4))
    b, near = oracle.lsh_hash(q, R)
    assert (b == 0).all() and near.all()


# --------------------------------------------------------------------------
# P3: the sort is the stable order by (bucket, position)
# --------------------------------------------------------------------------
@pytest.mark.parametrize("n_buckets", [1, 7, 64, 1024])
def test_sort_invariants(oracle_lib, n_buckets):
    rng = _rng(n_buckets)
    L, n_r = 2048, 3
    buckets = rng.integers(0, n_buckets, size=(2, 3, L, n_r)).astype(np.int32)
    perm, undo = oracle.lsh_sort_permute(buckets)
    for b in range(2):
        for h in range(3):
            for r in range(n_r):
                p, u, key = perm[b, h, r], undo[b, h, r], buckets[b, h, :, r]
                assert np.array_equal(np.sort(p), np.arange(L))
                assert np.array_equal(u[p], np.arange(L))
                assert np.array_equal(p, np.argsort(key, kind="stable"))
                composite = key[p].astype(np.int64) * L + p
                assert (np.diff(composite) > 0).all()


# --------------------------------------------------------------------------
# P4: multi-round union == attention over the union of buckets, each key once
# --------------------------------------------------------------------------
def union_attention(q, v, buckets, causal, scale):
    """Attention of i over T_i = {j != i : h^(r)(q_j) = h^(r)(q_i) for some r}
    (eq. union-pairs), each j once; O_i = v_i when T_i is empty."""
    L = q.shape[0]
    k = _keys(q)
    out = np.empty_like(v)
    for i in range(L):
        T = [j for j in range(L) if j != i and (buckets[j] == buckets[i]).any()
             and (not causal or j < i)]
        if not T:
            out[i] = v[i]
            continue
        a = np.array([scale * q[i] @ k[j] for j in T])
        w = np.exp(a - a.max())
        out[i] = (w / w.sum()) @ v[T]
    return out


@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("n_rounds,n_buckets", [(2, 2), (3, 4), (4, 8), (2, 8)])
def test_union_equivalence(oracle_lib, causal, n_rounds, n_buckets):
    """App. A: the N_ij term makes the rounds add up to the union exactly."""
    rng = _rng(100 * n_rounds + n_buckets + causal)
    L, d = 96, 16
    q = rng.standard_normal((L, d))
    v = rng.standard_normal((L, d))
    R = rng.standard_normal((n_rounds, d, n_buckets // 2))
    buckets, _ = oracle.lsh_hash(q.reshape(1, 1, L, d), R)
    b = buckets[0, 0]
    out, _, _ = run_oracle(q, v, b, chunk=L, causal=causal)
    want = union_attention(q, v, b, causal, 1.0 / np.sqrt(d))
    np.testing.assert_allclose(out, want, atol=1e-10, rtol=0)


def test_union_equivalence_causal_small_buckets(oracle_lib):
    """With causal masking and every bucket no larger than m, P_i lies inside
    P~_i (Sec. 2, 'If max |P_i| < m then P_i is a subset of P~_i'), so the
    chunked result still equals attention over the union."""
    rng = _rng(5)
    L, d, m, n_rounds = 256, 16, 16, 3
    q = rng.standard_normal((L, d))
    v = rng.standard_normal((L, d))
    # bucket ids with every bucket holding at most m tokens in every round
    b = np.stack([rng.permutation(np.arange(L) % (L // 12)) for _ in range(n_rounds)], 1)
    assert max(np.bincount(b[:, r]).max() for r in range(n_rounds)) <= m
    out, _, _ = run_oracle(q, v, b.astype(np.int32), chunk=m, causal=True)
    want = union_attention(q, v, b, True, 1.0 / np.sqrt(d))
    np.testing.assert_allclose(out, want, atol=1e-10, rtol=0)


# --------------------------------------------------------------------------
# P5: duplicated rounds collapse to one round (log N cancels)
# --------------------------------------------------------------------------
@pytest.mark.parametrize("causal", [False, True])
def test_duplicated_rounds(oracle_lib, causal):
    rng = _rng(21 + causal)
    L, d, n_b, m = 512, 32, 16, 32
    q = rng.standard_normal((1, 1, L, d))
    v = rng.standard_normal((1, 1, L, d))
    R1 = rng.standard_normal((1, d, n_b // 2))
    one = oracle.lsh_attention_fwd(q, v, R1, m, causal)
    for n_r in (2, 3, 5):
        many = oracle.lsh_attention_fwd(q, v, np.repeat(R1, n_r, axis=0), m, causal)
        np.testing.assert_allclose(many["out"], one["out"], atol=1e-10, rtol=0)
        # a row with other targets keeps its partition function (each round
        # carries log N = log n_r); a row left with only itself gains log n_r
        alone = one["lse"] < -1e4
        want = np.where(alone, one["lse"] + np.log(n_r), one["lse"])
        np.testing.assert_allclose(many["lse"], want, atol=1e-9, rtol=0)


# --------------------------------------------------------------------------
# P6: chunked oracle == dense evaluation of App. A with window masks
# --------------------------------------------------------------------------
@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("L,m,n_b,n_r,clustered", [(128, 16, 4, 2, False), (256, 32, 8, 3, True),
                                                  (192, 64, 2, 1, False), (256, 16, 16, 4, True),
                                                  (100, 16, 4, 2, True), (203, 32, 4, 3, False)])
def test_dense_windowed(oracle_lib, causal, L, m, n_b, n_r, clustered):
    """Buckets overflow past m here (few buckets, clustered inputs), so keys
    outside the window are really dropped.  In the last two cases m does not
    divide L: the dense form's chunk of a slot is floor(slot / m) with no
    padding, so its last chunk is the partial one."""
    rng = _rng(L + m + n_b + n_r + causal)
    d = 16
    if clustered:
        centres = rng.standard_normal((4, d))
        q = centres[rng.integers(0, 4, L)] + 0.3 * rng.standard_normal((L, d))
    else:
        q = rng.standard_normal((L, d))
    v = rng.standard_normal((L, d))
    R = rng.standard_normal((n_r, d, n_b // 2))
    buckets, _ = oracle.lsh_hash(q.reshape(1, 1, L, d), R)
    b = buckets[0, 0]
    assert max(np.bincount(b[:, r]).max() for r in range(n_r)) > m or n_b <= 2
    out, lse, _ = run_oracle(q, v, b, chunk=m, causal=causal)
    want, zwant = dense_output(q, v, b, m, causal, 1.0 / np.sqrt(d))
    np.testing.assert_allclose(out, want, atol=1e-10, rtol=0)
    np.testing.assert_allclose(lse, zwant, atol=1e-9, rtol=1e-13)


# --------------------------------------------------------------------------
# P7: tokens with no target but themselves return their own value
# --------------------------------------------------------------------------
def test_self_only_rows(oracle_lib):
    rng = _rng(7)
    L, d, n_r, m = 128, 16, 3, 32
    q = rng.standard_normal((L, d))
    v = rng.standard_normal((L, d))
    b = rng.integers(0, 4, size=(L, n_r)).astype(np.int32)
    lonely = [5, 77]
    for r in range(n_r):
        for t, i in enumerate(lonely):
            b[i, r] = 10 + t  # alone in its bucket in every round
    for causal in (False, True):
        out, lse, _ = run_oracle(q, v, b, chunk=m, causal=causal)
        # the round weights exp(z_r - z) are formed from z ~ -1e5, whose fp64
        # spacing is ~1.5e-11, so the fallback is exact only to that level
        for i in lonely:
            np.testing.assert_allclose(out[i], v[i], atol=1e-10, rtol=0)
        if causal:
            np.testing.assert_allclose(out[0], v[0], atol=1e-10, rtol=0)


# --------------------------------------------------------------------------
# P10: with one round the combine step is the identity up to the sort
# --------------------------------------------------------------------------
def test_single_round_combine_identity(oracle_lib):
    rng = _rng(9)
    L, d = 256, 64
    q = rng.standard_normal((2, 2, L, d))
    v = rng.standard_normal((2, 2, L, d))
    R = rng.standard_normal((1, d, 8))
    res = oracle.lsh_attention_fwd(q, v, R, 64, False)
    for b in range(2):
        for h in range(2):
            u = res["undo"][b, h, 0]
            assert np.array_equal(res["out"][b, h], res["o_rounds"][b, h, 0][u])
            assert np.array_equal(res["lse"][b, h], res["lse_rounds"][b, h, 0][u])


# --------------------------------------------------------------------------
# P8: backward against fp64 autograd and finite differences
# --------------------------------------------------------------------------
def torch_dense_loss(q, v, dout, buckets, chunk, causal, scale, self_mask=1e5, after=0,
                     across=False):
    """sum(dO * O) with O the dense App. A output, differentiable in q and v."""
    L, d = q.shape
    n_r = buckets.shape[1]
    k = q / q.norm(dim=1, keepdim=True)
    pos = np.arange(L)
    win = window_masks(buckets, chunk, after)
    if across:
        N = sum(w.astype(np.int64) for w in win)
    else:
        N = (buckets[:, None, :] == buckets[None, :, :]).sum(-1)
    with np.errstate(divide="ignore"):
        M = np.where(np.eye(L, dtype=bool), self_mask, np.log(N.astype(np.float64)))
    M = torch.from_numpy(M)
    logits = []
    for r in range(n_r):
        ok = win[r].copy()
        if not across:
            ok &= buckets[:, r][:, None] == buckets[:, r][None, :]
        if causal:
            ok &= pos[None, :] <= pos[:, None]
        a = scale * (q @ k.T) - M
        logits.append(torch.where(torch.from_numpy(ok), a, torch.full_like(a, -torch.inf)))
    flat = torch.cat(logits, dim=1)
    w = torch.softmax(flat, dim=1)
    out = w @ v.repeat(n_r, 1)
    return (out * dout).sum(), out


@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("n_r,n_b,m,L", [(1, 4, 16, 128), (3, 8, 16, 128), (4, 4, 32, 128),
                                         (3, 8, 32, 113)])
def test_backward_autograd(oracle_lib, causal, n_r, n_b, m, L):
    """The last case has a partial last chunk (m does not divide L)."""
    rng = _rng(31 + n_r + n_b + causal + L)
    d = 16
    q = rng.standard_normal((L, d))
    v = rng.standard_normal((L, d))
    dout = rng.standard_normal((L, d))
    R = rng.standard_normal((n_r, d, n_b // 2))
    buckets, _ = oracle.lsh_hash(q.reshape(1, 1, L, d), R)
    b = buckets[0, 0]
    scale = 1.0 / np.sqrt(d)
    qt = torch.tensor(q, requires_grad=True)
    vt = torch.tensor(v, requires_grad=True)
    loss, out_t = torch_dense_loss(qt, vt, torch.tensor(dout), b, m, causal, scale)
    loss.backward()
    out, lse, _ = run_oracle(q, v, b, chunk=m, causal=causal)
    np.testing.assert_allclose(out, out_t.detach().numpy(), atol=1e-10, rtol=0)
    dq, dv = oracle.lsh_chunk_attn_bwd(q.reshape(1, 1, L, d), v.reshape(1, 1, L, d),
                                       out.reshape(1, 1, L, d), dout.reshape(1, 1, L, d),
                                       lse.reshape(1, 1, L), buckets,
                                       oracle.lsh_sort_permute(buckets)[0], m, causal)
    np.testing.assert_allclose(dq[0, 0], qt.grad.numpy(), atol=1e-10, rtol=0)
    np.testing.assert_allclose(dv[0, 0], vt.grad.numpy(), atol=1e-10, rtol=0)


def test_backward_finite_differences(oracle_lib):
    rng = _rng(44)
    L, d, n_r, n_b, m = 96, 8, 2, 4, 16
    q = rng.standard_normal((L, d))
    v = rng.standard_normal((L, d))
    dout = rng.standard_normal((L, d))
    R = rng.standard_normal((n_r, d, n_b // 2))
    buckets, _ = oracle.lsh_hash(q.reshape(1, 1, L, d), R)
    b = buckets[0, 0]
    out, lse, _ = run_oracle(q, v, b, chunk=m, causal=True)
    dq, dv = oracle.lsh_chunk_attn_bwd(q[None, None], v[None, None], out[None, None],
                                       dout[None, None], lse[None, None], buckets,
                                       oracle.lsh_sort_permute(buckets)[0], m, True)

    def loss(qq, vv):
        o, _, _ = run_oracle(qq, vv, b, chunk=m, causal=True)
        return float((o * dout).sum())

    h = 1e-6
    for _ in range(8):
        i, t = rng.integers(0, L), rng.integers(0, d)
        e = np.zeros((L, d))
        e[i, t] = h
        fd_q = (loss(q + e, v) - loss(q - e, v)) / (2 * h)
        fd_v = (loss(q, v + e) - loss(q, v - e)) / (2 * h)
        assert abs(fd_q - dq[0, 0, i, t]) < 1e-6 * max(1.0, abs(fd_q))
        assert abs(fd_v - dv[0, 0, i, t]) < 1e-6 * max(1.0, abs(fd_v))


# --------------------------------------------------------------------------
# argument checks of the oracle library itself
# --------------------------------------------------------------------------
def test_oracle_rejects_bad_arguments(oracle_lib):
    q = np.zeros((1, 1, 64, 8))
    with pytest.raises(RuntimeError):
        oracle.lsh_hash(q, np.zeros((1, 8, 0)))  # n_buckets = 0
    with pytest.raises(RuntimeError):
        oracle.lsh_chunk_attn_fwd(q, q, np.zeros((1, 1, 64, 1), np.int32),
                                  np.zeros((1, 1, 1, 64), np.int32), 0, False)  # m = 0


# --------------------------------------------------------------------------
# The dense baseline (full shared-QK attention, Sec. 2 memory-efficient
# attention): pinned to the LSH oracle's one-bucket case, to PyTorch's
# attention routine, and to its special cases
# --------------------------------------------------------------------------
@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("L,d", [(64, 8), (100, 64), (203, 16)])
def test_dense_is_one_bucket_one_chunk(oracle_lib, causal, L, d):
    """With every token in one bucket, one round and a chunk holding the whole
    sequence, the LSH window covers all keys: the two oracle functions (no
    shared code beyond the row norms) must agree."""
    rng = _rng(7 * L + d + causal)
    q = rng.standard_normal((L, d))
    v = rng.standard_normal((L, d))
    out_l, lse_l, _ = run_oracle(q, v, np.zeros((L, 1), np.int32), chunk=L, causal=causal)
    out_d, lse_d = oracle.dense_attn_fwd(q.reshape(1, 1, L, d), v.reshape(1, 1, L, d), causal)
    np.testing.assert_allclose(out_d[0, 0], out_l, atol=1e-12, rtol=0)
    np.testing.assert_allclose(lse_d[0, 0], lse_l, atol=1e-9, rtol=0)


@pytest.mark.parametrize("causal", [False, True])
def test_dense_matches_torch_attention(oracle_lib, causal):
    """PyTorch's scaled_dot_product_attention (CPU, float64) with K = Q/|Q|
    and the App. A masks as an additive float mask: -1e5 on the diagonal,
    -inf above it under causal masking."""
    B, H, L, d = 2, 3, 96, 64
    rng = _rng(11 + causal)
    q = rng.standard_normal((B, H, L, d)) * rng.uniform(0.5, 3.0, (B, H, L, 1))
    v = rng.standard_normal((B, H, L, d))
    out, _ = oracle.dense_attn_fwd(q, v, causal)
    qt, vt = torch.from_numpy(q), torch.from_numpy(v)
    kt = qt / qt.norm(dim=-1, keepdim=True)
    mask = torch.zeros((L, L), dtype=torch.float64)
    mask.fill_diagonal_(-1e5)
    if causal:
        mask = mask.masked_fill(torch.ones((L, L), dtype=torch.bool).triu(1), float("-inf"))
    ref = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, attn_mask=mask,
                                                           scale=1.0 / np.sqrt(d))
    np.testing.assert_allclose(out, ref.numpy(), atol=1e-12, rtol=0)


def test_dense_special_cases(oracle_lib):
    """Causal: the first token's only key is itself (output v_0, log-partition
    scale*|q_0| - 1e5).  A zero query has k = 0 (logit 0 as a key) and, as a
    query, weighs every other key equally.  Non-causal attention is
    equivariant under a permutation of the positions."""
    L, d = 40, 16
    rng = _rng(5)
    q = rng.standard_normal((L, d))
    v = rng.standard_normal((L, d))
    q[7] = 0.0
    scale = 1.0 / np.sqrt(d)
    out_c, lse_c = oracle.dense_attn_fwd(q.reshape(1, 1, L, d), v.reshape(1, 1, L, d), True)
    assert np.array_equal(out_c[0, 0, 0], v[0])
    assert abs(lse_c[0, 0, 0] - (scale * np.linalg.norm(q[0]) - 1e5)) < 1e-9
    out, lse = oracle.dense_attn_fwd(q.reshape(1, 1, L, d), v.reshape(1, 1, L, d), False)
    others = np.delete(np.arange(L), 7)
    np.testing.assert_allclose(out[0, 0, 7], v[others].mean(0), atol=1e-12, rtol=0)
    assert abs(lse[0, 0, 7] - np.log(L - 1)) < 1e-12
    p = rng.permutation(L)
    out_p, lse_p = oracle.dense_attn_fwd(q[p].reshape(1, 1, L, d), v[p].reshape(1, 1, L, d), False)
    np.testing.assert_allclose(out_p[0, 0], out[0, 0][p], atol=1e-12, rtol=0)
    np.testing.assert_allclose(lse_p[0, 0], lse[0, 0][p], atol=1e-12, rtol=0)


@pytest.mark.parametrize("causal", [False, True])
def test_dense_selected_rows(oracle_lib, causal):
    """The row-sampled form (used at full size) returns the same rows as the
    whole computation, in the order asked for, across batch and head."""
    B, H, L, d = 2, 2, 70, 8
    rng = _rng(23 + causal)
    q = rng.standard_normal((B, H, L, d))
    v = rng.standard_normal((B, H, L, d))
    out, lse = oracle.dense_attn_fwd(q, v, causal)
    rows = np.array([0, 69, 70, 139, 215, 3 * L + 5, 4 * L - 1, 71])
    o_s, l_s = oracle.dense_attn_fwd(q, v, causal, rows=rows)
    assert np.array_equal(o_s, out.reshape(-1, d)[rows])
    assert np.array_equal(l_s, lse.reshape(-1)[rows])



# --------------------------------------------------------------------------
# Variants (off by default; the paper does not spell them out): a look-ahead
# chunk, attending across buckets, one R per head.  Each is pinned to a dense
# or brute-force form that shares nothing with the oracle's loops.
# --------------------------------------------------------------------------
def _clustered(rng, L, d, k=4):
    centres = rng.standard_normal((k, d))
    return centres[rng.integers(0, k, L)] + 0.3 * rng.standard_normal((L, d))


@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("after,across", [(1, False), (0, True), (1, True)])
@pytest.mark.parametrize("L,m,n_b,n_r", [(128, 16, 4, 2), (203, 32, 8, 3), (256, 16, 16, 4)])
def test_variants_dense_windowed(oracle_lib, causal, after, across, L, m, n_b, n_r):
    """The chunk loops with a look-ahead and/or attention across buckets equal
    the dense evaluation of App. A with those windows and target sets (the
    P6 form), with buckets overflowing m and a partial last chunk."""
    rng = _rng(L + m + n_b + n_r + causal + 10 * after + 20 * across)
    d = 16
    q = _clustered(rng, L, d)
    v = rng.standard_normal((L, d))
    R = rng.standard_normal((n_r, d, n_b // 2))
    b = oracle.lsh_hash(q.reshape(1, 1, L, d), R)[0][0, 0]
    out, lse, _ = run_oracle(q, v, b, chunk=m, causal=causal, after=after, across=across)
    want, zwant = dense_output(q, v, b, m, causal, 1.0 / np.sqrt(d), after=after, across=across)
    np.testing.assert_allclose(out, want, atol=1e-10, rtol=0)
    np.testing.assert_allclose(lse, zwant, atol=1e-9, rtol=1e-13)


def test_lookahead_covers_small_buckets_non_causal(oracle_lib):
    """Without causal masking P~ misses the part of a bucket that spills into
    the next chunk, so the rounds do not add up to attention over the union of
    buckets even when every bucket holds at most m tokens; one look-ahead
    chunk closes that gap (Sec. 2, 'If max |P_i| < m then P_i is a subset of
    P~_i')."""
    rng = _rng(6)
    L, d, m, n_rounds = 256, 16, 16, 3
    q = rng.standard_normal((L, d))
    v = rng.standard_normal((L, d))
    b = np.stack([rng.permutation(np.arange(L) % (L // 12)) for _ in range(n_rounds)], 1)
    b = b.astype(np.int32)
    assert max(np.bincount(b[:, r]).max() for r in range(n_rounds)) <= m
    want = union_attention(q, v, b, False, 1.0 / np.sqrt(d))
    plain, _, _ = run_oracle(q, v, b, chunk=m, causal=False)
    ahead, _, _ = run_oracle(q, v, b, chunk=m, causal=False, after=1)
    assert np.abs(plain - want).max() > 1e-3  # the gap is real
    np.testing.assert_allclose(ahead, want, atol=1e-10, rtol=0)


@pytest.mark.parametrize("causal", [False, True])
def test_across_one_chunk_is_dense(oracle_lib, causal):
    """Across buckets with one chunk spanning the sequence every round's
    target set is every key, N_ij = n_rounds for every pair and the output is
    dense self-masked shared-QK attention (eq. attn with k = q/|q|) whatever
    the bucket ids."""
    rng = _rng(61 + causal)
    L, d, n_r = 96, 16, 3
    q = rng.standard_normal((L, d))
    v = rng.standard_normal((L, d))
    b = rng.integers(0, 8, size=(L, n_r)).astype(np.int32)
    out, _, _ = run_oracle(q, v, b, chunk=L, causal=causal, across=True)
    k = _keys(q)
    a = q @ k.T / np.sqrt(d)
    ok = ~np.eye(L, dtype=bool)
    if causal:
        ok &= np.tri(L, dtype=bool)
    a = np.where(ok, a, -np.inf)
    want = np.empty_like(v)
    for i in range(L):
        if not ok[i].any():
            want[i] = v[i]
            continue
        w = np.exp(a[i] - a[i].max())
        want[i] = (w / w.sum()) @ v
    np.testing.assert_allclose(out, want, atol=1e-10, rtol=0)


@pytest.mark.parametrize("after,across", [(1, False), (0, True), (1, True)])
def test_variants_backward_autograd(oracle_lib, after, across):
    """The backward of the variants against fp64 autograd of the dense form."""
    rng = _rng(71 + after + 2 * across)
    L, d, n_r, n_b, m = 113, 16, 3, 8, 16
    for causal in (False, True):
        q = _clustered(rng, L, d)
        v = rng.standard_normal((L, d))
        dout = rng.standard_normal((L, d))
        R = rng.standard_normal((n_r, d, n_b // 2))
        buckets, _ = oracle.lsh_hash(q.reshape(1, 1, L, d), R)
        b = buckets[0, 0]
        scale = 1.0 / np.sqrt(d)
        qt = torch.tensor(q, requires_grad=True)
        vt = torch.tensor(v, requires_grad=True)
        loss, out_t = torch_dense_loss(qt, vt, torch.tensor(dout), b, m, causal, scale,
                                       after=after, across=across)
        loss.backward()
        out, lse, _ = run_oracle(q, v, b, chunk=m, causal=causal, after=after, across=across)
        np.testing.assert_allclose(out, out_t.detach().numpy(), atol=1e-10, rtol=0)
        dq, dv = oracle.lsh_chunk_attn_bwd(q[None, None], v[None, None], out[None, None],
                                           dout[None, None], lse[None, None], buckets,
                                           oracle.lsh_sort_permute(buckets)[0], m, causal,
                                           after=after, across=across)
        np.testing.assert_allclose(dq[0, 0], qt.grad.numpy(), atol=1e-10, rtol=0)
        np.testing.assert_allclose(dv[0, 0], vt.grad.numpy(), atol=1e-10, rtol=0)


def test_hash_per_head(oracle_lib):
    """One R per head: head h's ids are the brute-force argmax of
    [x R_h; -x R_h] (Sec. 2), and R repeated over the heads gives the ids of
    the shared R."""
    rng = _rng(81)
    B, H, L, d, n_r, n_b = 2, 3, 40, 16, 2, 16
    q = rng.standard_normal((B, H, L, d))
    Rh = rng.standard_normal((H, n_r, d, n_b // 2))
    got, _ = oracle.lsh_hash(q, Rh)
    for h in range(H):
        for r in range(n_r):
            p = q[:, h] @ Rh[h, r]
            want = np.argmax(np.concatenate([p, -p], axis=-1), axis=-1)
            assert np.array_equal(got[:, h, :, r], want)
    shared, _ = oracle.lsh_hash(q, Rh[0])
    same, _ = oracle.lsh_hash(q, np.repeat(Rh[:1], H, axis=0))
    assert np.array_equal(same, shared)
