"""The C ABI without a GPU: the library loads, exports every symbol the header
declares, sizes workspaces, and rejects bad arguments before any HIP call."""
import ctypes
import os
import re

import pytest

from paper_2001_04451_amd import lsh

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADERS = [os.path.join(ROOT, "include", h) for h in ("lsh.h", "lsh_block.h")]


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(lsh.LIB_PATH):
        pytest.skip("liblsh.so not built (run __graft_entry__.build())")
    return lsh.lib()


def declared_symbols():
    text = "".join(open(h).read() for h in HEADERS)
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(lsh_[a-z0-9_]+)\s*\(", text)))


def test_header_symbols_exported(L):
    names = declared_symbols()
    assert set(names) == set(lsh.EXPORTED)
    for name in names:
        assert hasattr(L, name), f"{name} missing from liblsh.so"


def test_status_strings(L):
    assert L.lsh_status_string(0) == b"ok"
    assert L.lsh_status_string(-1) == b"invalid argument"
    assert L.lsh_status_string(-2) == b"unsupported configuration"
    assert L.lsh_status_string(-3) == b"HIP runtime error"


def _cfg(**kw):
    base = dict(B=1, H=2, L=1024, d=64, n_buckets=64, n_rounds=2, chunk=64, causal=0,
                scale=0.125, self_mask=1e5)
    base.update(kw)
    return lsh.LshConfig(**base)


FAKE = ctypes.c_void_p(0x1000)  # never dereferenced: every call below fails validation


@pytest.mark.parametrize("bad", [dict(B=0), dict(L=0), dict(d=0), dict(n_buckets=7),
                                 dict(n_buckets=0), dict(n_rounds=0), dict(chunk=0),
                                 dict(H=0), dict(scale=float("nan"))])
def test_invalid_config(L, bad):
    c = _cfg(**bad)
    rc = L.lsh_hash(ctypes.byref(c), lsh.LSH_BF16, FAKE, FAKE, FAKE, FAKE, 1 << 30, None)
    assert rc == lsh.LSH_ERR_INVALID
    rc = L.lsh_chunk_attn_fwd(ctypes.byref(c), lsh.LSH_BF16, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE,
                              FAKE, FAKE, FAKE, FAKE, 1 << 30, None)
    assert rc == lsh.LSH_ERR_INVALID
    assert L.lsh_workspace_bytes(ctypes.byref(c), lsh.LSH_BF16, lsh.LSH_OP_FORWARD) == 0


def test_null_pointers_and_small_workspace(L):
    c = _cfg()
    assert L.lsh_hash(None, 1, FAKE, FAKE, FAKE, FAKE, 1 << 30, None) == lsh.LSH_ERR_INVALID
    assert L.lsh_hash(ctypes.byref(c), 1, None, FAKE, FAKE, FAKE, 1 << 30, None) == lsh.LSH_ERR_INVALID
    need = L.lsh_workspace_bytes(ctypes.byref(c), 1, lsh.LSH_OP_HASH)
    assert need > 0
    assert L.lsh_hash(ctypes.byref(c), 1, FAKE, FAKE, FAKE, FAKE, need - 1, None) == lsh.LSH_ERR_INVALID
    assert L.lsh_hash(ctypes.byref(c), 7, FAKE, FAKE, FAKE, FAKE, need, None) == lsh.LSH_ERR_INVALID
    assert L.lsh_sort_permute(ctypes.byref(c), FAKE, None, FAKE, FAKE, FAKE, 1 << 30, None) == lsh.LSH_ERR_INVALID
    assert L.lsh_combine_rounds(ctypes.byref(c), 1, FAKE, FAKE, FAKE, None, FAKE, None,
                                None) == lsh.LSH_ERR_INVALID
    # bf16 calls need the per-row exponents of the fp16 rows; fp32 calls do not
    assert L.lsh_combine_rounds(ctypes.byref(c), 1, FAKE, None, FAKE, FAKE, FAKE, None,
                                None) == lsh.LSH_ERR_INVALID
    fwd = L.lsh_workspace_bytes(ctypes.byref(c), 1, lsh.LSH_OP_FORWARD)
    assert L.lsh_attention_fwd(ctypes.byref(c), 1, FAKE, FAKE, FAKE, FAKE, None, FAKE, FAKE, FAKE,
                               FAKE, FAKE, fwd - 1, None) == lsh.LSH_ERR_INVALID
    # bf16 attention needs its per-token workspace; fp32 needs none
    attn = L.lsh_workspace_bytes(ctypes.byref(c), 1, lsh.LSH_OP_ATTN_FWD)
    assert attn > 0 and L.lsh_workspace_bytes(ctypes.byref(c), 0, lsh.LSH_OP_ATTN_FWD) == 0
    assert L.lsh_chunk_attn_fwd(ctypes.byref(c), 1, FAKE, FAKE, FAKE, FAKE, None, FAKE, FAKE,
                                FAKE, FAKE, FAKE, attn - 1, None) == lsh.LSH_ERR_INVALID
    assert L.lsh_chunk_attn_fwd(ctypes.byref(c), 1, FAKE, FAKE, FAKE, FAKE, None, FAKE, FAKE,
                                FAKE, FAKE, None, attn, None) == lsh.LSH_ERR_INVALID
    assert L.lsh_chunk_attn_fwd(ctypes.byref(c), 1, FAKE, FAKE, FAKE, FAKE, None, FAKE, FAKE,
                                None, FAKE, FAKE, attn, None) == lsh.LSH_ERR_INVALID


@pytest.mark.parametrize("unsup", [dict(d=32), dict(chunk=96, L=1056), dict(n_buckets=2048),
                                   dict(n_rounds=17)])
def test_unsupported_shapes(L, unsup):
    c = _cfg(**unsup)
    need = L.lsh_workspace_bytes(ctypes.byref(c), 1, lsh.LSH_OP_FORWARD)
    rc = L.lsh_attention_fwd(ctypes.byref(c), 1, FAKE, FAKE, FAKE, FAKE, None, FAKE, FAKE, FAKE,
                             FAKE, FAKE, need, None)
    assert rc == lsh.LSH_ERR_UNSUPPORTED


def test_backward_is_bf16_only(L):
    c = _cfg()
    need = L.lsh_workspace_bytes(ctypes.byref(c), lsh.LSH_F32, lsh.LSH_OP_ATTN_BWD)
    rc = L.lsh_chunk_attn_bwd(ctypes.byref(c), lsh.LSH_F32, *([FAKE] * 12), need, None)
    assert rc == lsh.LSH_ERR_UNSUPPORTED


def test_workspace_sizes(L):
    c = _cfg(B=1, H=16, L=65536, n_buckets=1024, n_rounds=8)
    rr = 16 * 65536 * 8
    # per-round outputs (fp16 rows and their exponent bytes for bf16 calls, fp32
    # rows for fp32 calls) plus fp32 log-partitions
    fwd = L.lsh_workspace_bytes(ctypes.byref(c), 1, lsh.LSH_OP_FORWARD)
    assert fwd >= rr * 64 * 2 + rr + rr * 4
    fwd32 = L.lsh_workspace_bytes(ctypes.byref(c), 0, lsh.LSH_OP_FORWARD)
    assert fwd32 >= rr * 64 * 4 + rr * 4
    assert L.lsh_workspace_bytes(ctypes.byref(c), 0, lsh.LSH_OP_ATTN_FWD) == 0


def test_product_never_touches_the_oracle():
    """The GPU package imports, links and includes nothing from oracle/."""
    pkg = os.path.join(ROOT, "paper_2001_04451_amd")
    for dirpath, _, files in os.walk(pkg):
        for f in files:
            if f.endswith((".py", ".hip", ".cpp", ".h")):
                text = open(os.path.join(dirpath, f)).read()
                assert not re.search(r"^\s*(import|from)\s+oracle", text, re.M), f
                assert "lsh_oracle" not in text and "lsh_ref_" not in text, f


def test_dense_entry_validation(L):
    """The dense baseline reads only the shape, causal flag and scales; its
    errors come back before any HIP call."""
    c = _cfg(n_buckets=0, n_rounds=0, chunk=0)  # hashing fields are not read
    need = L.lsh_workspace_bytes(ctypes.byref(c), lsh.LSH_BF16, lsh.LSH_OP_DENSE_FWD)
    assert need >= c.B * c.H * c.L * 4
    args = (FAKE, FAKE, FAKE, None, FAKE)
    assert L.lsh_dense_attn_fwd(None, lsh.LSH_BF16, *args, need, None) == lsh.LSH_ERR_INVALID
    assert L.lsh_dense_attn_fwd(ctypes.byref(c), lsh.LSH_BF16, *args, need - 1, None) == lsh.LSH_ERR_INVALID
    assert L.lsh_dense_attn_fwd(ctypes.byref(c), lsh.LSH_BF16, None, FAKE, FAKE, None, FAKE, need,
                                None) == lsh.LSH_ERR_INVALID
    assert L.lsh_dense_attn_fwd(ctypes.byref(c), lsh.LSH_BF16, FAKE, FAKE, FAKE, None, None, need,
                                None) == lsh.LSH_ERR_INVALID
    assert L.lsh_dense_attn_fwd(ctypes.byref(c), 5, *args, need, None) == lsh.LSH_ERR_INVALID
    assert L.lsh_dense_attn_fwd(ctypes.byref(c), lsh.LSH_F32, *args, 1 << 30, None) == lsh.LSH_ERR_UNSUPPORTED
    c32 = _cfg(d=32)
    assert L.lsh_dense_attn_fwd(ctypes.byref(c32), lsh.LSH_BF16, *args, 1 << 30, None) == lsh.LSH_ERR_UNSUPPORTED
    bad = _cfg(L=0)
    assert L.lsh_workspace_bytes(ctypes.byref(bad), lsh.LSH_BF16, lsh.LSH_OP_DENSE_FWD) == 0
    assert L.lsh_dense_attn_fwd(ctypes.byref(bad), lsh.LSH_BF16, *args, 1 << 30, None) == lsh.LSH_ERR_INVALID


def test_chunk_lengths(L):
    """Chunks of 64 or 128 on the forward (other lengths unsupported); the
    backward takes chunks of 64 only."""
    c128 = _cfg(chunk=128)
    for dtype in (lsh.LSH_BF16, lsh.LSH_F32):
        bwd = L.lsh_workspace_bytes(ctypes.byref(c128), dtype, lsh.LSH_OP_ATTN_BWD)
        assert L.lsh_chunk_attn_bwd(ctypes.byref(c128), dtype, *([FAKE] * 12), bwd,
                                    None) == lsh.LSH_ERR_UNSUPPORTED
    c96 = _cfg(chunk=96)
    for dtype in (lsh.LSH_BF16, lsh.LSH_F32):
        assert L.lsh_chunk_attn_fwd(ctypes.byref(c96), dtype, FAKE, FAKE, FAKE, FAKE, None, FAKE,
                                    FAKE, FAKE, FAKE, FAKE, 1 << 30, None) == lsh.LSH_ERR_UNSUPPORTED


@pytest.mark.parametrize("self_mask", [0.0, 10.0, -1e5, 9999.0])
def test_self_mask_below_bound(L, self_mask):
    """The attention calls drop a token's own key whenever it has another target,
    which is exact only for a large self mask (App. A uses 1e5): below 1e4 they
    refuse the configuration before any HIP call.  Hash and sort do not read
    self_mask and accept it."""
    c = _cfg(self_mask=self_mask)
    bf = lsh.LSH_BF16
    fwd = L.lsh_workspace_bytes(ctypes.byref(c), bf, lsh.LSH_OP_FORWARD)
    assert L.lsh_attention_fwd(ctypes.byref(c), bf, FAKE, FAKE, FAKE, FAKE, None, FAKE, FAKE, FAKE,
                               FAKE, FAKE, fwd, None) == lsh.LSH_ERR_UNSUPPORTED
    attn = L.lsh_workspace_bytes(ctypes.byref(c), bf, lsh.LSH_OP_ATTN_FWD)
    assert L.lsh_chunk_attn_fwd(ctypes.byref(c), bf, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE,
                                FAKE, FAKE, attn, None) == lsh.LSH_ERR_UNSUPPORTED
    bwd = L.lsh_workspace_bytes(ctypes.byref(c), bf, lsh.LSH_OP_ATTN_BWD)
    assert L.lsh_chunk_attn_bwd(ctypes.byref(c), bf, *([FAKE] * 12), bwd, None) == lsh.LSH_ERR_UNSUPPORTED
    dense = L.lsh_workspace_bytes(ctypes.byref(c), bf, lsh.LSH_OP_DENSE_FWD)
    assert L.lsh_dense_attn_fwd(ctypes.byref(c), bf, FAKE, FAKE, FAKE, None, FAKE, dense,
                                None) == lsh.LSH_ERR_UNSUPPORTED
    # hash with an undersized workspace: INVALID (validation reached), not UNSUPPORTED
    assert L.lsh_hash(ctypes.byref(c), bf, FAKE, FAKE, FAKE, FAKE, 0, None) == lsh.LSH_ERR_INVALID


def test_backward_alignment(L):
    """The backward moves rows in 16-byte pieces: a misaligned q, v, out, dout,
    dq, dv or workspace is refused before any HIP call."""
    c = _cfg()
    bf = lsh.LSH_BF16
    need = L.lsh_workspace_bytes(ctypes.byref(c), bf, lsh.LSH_OP_ATTN_BWD)
    odd = ctypes.c_void_p(0x1008)
    # pointer arguments: q, v, out, dout, lse_total, buckets, perm, undo,
    # bucket_start, dq, dv, workspace
    for k in (0, 1, 2, 3, 9, 10, 11):
        args = [FAKE] * 12
        args[k] = odd
        rc = L.lsh_chunk_attn_bwd(ctypes.byref(c), bf, *args, need, None)
        assert rc == lsh.LSH_ERR_INVALID, k
    assert L.lsh_chunk_attn_bwd(ctypes.byref(c), bf, *([FAKE] * 12), 0, None) == lsh.LSH_ERR_INVALID



@pytest.mark.parametrize("variant", [dict(chunks_after=1), dict(attend_across=1),
                                     dict(chunks_after=2)])
def test_variant_support(L, variant):
    """Look-ahead and attention across buckets: the fp32 forward takes both
    (one look-ahead chunk at most), the bf16 forward the look-ahead; the rest
    and the backward refuse them before any HIP call; a negative look-ahead is
    invalid."""
    c = _cfg(**variant)
    for dtype in (lsh.LSH_BF16, lsh.LSH_F32):
        supported = variant.get("chunks_after", 0) <= 1 and (
            dtype == lsh.LSH_F32 or not variant.get("attend_across", 0))
        if supported:
            continue  # would launch: not called without a GPU
        fwd = L.lsh_workspace_bytes(ctypes.byref(c), dtype, lsh.LSH_OP_FORWARD)
        rc = L.lsh_attention_fwd(ctypes.byref(c), dtype, FAKE, FAKE, FAKE, FAKE, None, FAKE, FAKE,
                                 FAKE, FAKE, FAKE, fwd, None)
        assert rc == lsh.LSH_ERR_UNSUPPORTED
    bwd = L.lsh_workspace_bytes(ctypes.byref(c), lsh.LSH_BF16, lsh.LSH_OP_ATTN_BWD)
    assert L.lsh_chunk_attn_bwd(ctypes.byref(c), lsh.LSH_BF16, *([FAKE] * 12), bwd,
                                None) == lsh.LSH_ERR_UNSUPPORTED
    neg = _cfg(chunks_after=-1)
    assert L.lsh_workspace_bytes(ctypes.byref(neg), lsh.LSH_F32, lsh.LSH_OP_FORWARD) == 0


def test_across_needs_undo(L):
    c = _cfg(attend_across=1)
    assert L.lsh_chunk_attn_fwd(ctypes.byref(c), lsh.LSH_F32, FAKE, FAKE, FAKE, FAKE, None, FAKE,
                                FAKE, None, FAKE, None, 0, None) == lsh.LSH_ERR_INVALID


def _bcfg(attn=None, d_ff=256, ff_chunk=0, ln_eps=1e-5):
    attn = attn or _cfg(B=1, H=2, L=256, n_buckets=16, n_rounds=2, causal=1)
    return lsh.BlockConfigC(attn, d_ff, ff_chunk, ln_eps)


def _bweights(**kw):
    names = [n for n, _ in lsh.BlockWeightsC._fields_]
    vals = {n: FAKE.value for n in names}
    vals.update(kw)
    return lsh.BlockWeightsC(**vals)


def test_block_workspace_and_validation(L):
    """The reversible block's entry points validate before any HIP call."""
    c = _bcfg()
    for op in (lsh.LSH_BLOCK_OP_ATTN, lsh.LSH_BLOCK_OP_FF, lsh.LSH_BLOCK_OP_BLOCK):
        assert L.lsh_block_workspace_bytes(ctypes.byref(c), op) > 0
    assert L.lsh_block_workspace_bytes(None, 0) == 0
    # the feed-forward's scratch follows its chunk
    big = L.lsh_block_workspace_bytes(ctypes.byref(_bcfg(ff_chunk=0)), lsh.LSH_BLOCK_OP_FF)
    small = L.lsh_block_workspace_bytes(ctypes.byref(_bcfg(ff_chunk=64)), lsh.LSH_BLOCK_OP_FF)
    assert small < big
    w = _bweights()
    huge = 1 << 40

    def att(cfg, wts, ws_bytes=huge, x=FAKE):
        return L.lsh_rev_attention(ctypes.byref(cfg), ctypes.byref(wts) if wts else None, x, None, FAKE,
                                   1.0, FAKE, ws_bytes, None)

    def ff(cfg, wts, ws_bytes=huge):
        return L.lsh_rev_feed_forward(ctypes.byref(cfg), ctypes.byref(wts) if wts else None, FAKE, None, FAKE,
                                      1.0, FAKE, ws_bytes, None)

    assert att(_bcfg(d_ff=0), w) == lsh.LSH_ERR_INVALID
    assert att(_bcfg(d_ff=100), w) == lsh.LSH_ERR_UNSUPPORTED
    assert att(_bcfg(attn=_cfg(B=1, H=3, L=256, n_buckets=16, n_rounds=2)), w) == lsh.LSH_ERR_UNSUPPORTED
    assert att(_bcfg(attn=_cfg(B=1, H=2, L=256, n_buckets=16, n_rounds=2, d=32)), w) == lsh.LSH_ERR_UNSUPPORTED
    assert att(_bcfg(ln_eps=float("nan")), w) == lsh.LSH_ERR_INVALID
    assert att(c, None) == lsh.LSH_ERR_INVALID
    assert att(c, _bweights(w_qk=None)) == lsh.LSH_ERR_INVALID
    assert att(c, _bweights(w_o=FAKE.value + 4)) == lsh.LSH_ERR_INVALID  # misaligned
    assert att(c, w, ws_bytes=16) == lsh.LSH_ERR_INVALID
    assert att(c, w, x=None) == lsh.LSH_ERR_INVALID
    assert ff(c, _bweights(b2=None)) == lsh.LSH_ERR_INVALID
    assert ff(c, w, ws_bytes=16) == lsh.LSH_ERR_INVALID
    for fn in (L.lsh_rev_block_fwd, L.lsh_rev_block_inv):
        assert fn(ctypes.byref(c), ctypes.byref(w), FAKE, FAKE, FAKE, None, FAKE, huge, None) == lsh.LSH_ERR_INVALID
        assert fn(ctypes.byref(c), ctypes.byref(w), FAKE, FAKE, FAKE, FAKE, FAKE, 16, None) == lsh.LSH_ERR_INVALID


def test_linear_validation(L):
    f = L.lsh_linear_bf16
    assert f(128, 100, 64, FAKE, FAKE, None, None, 1.0, FAKE, None, None) == lsh.LSH_ERR_UNSUPPORTED
    assert f(128, 128, 32, FAKE, FAKE, None, None, 1.0, FAKE, None, None) == lsh.LSH_ERR_UNSUPPORTED
    assert f(128, 128, 64, None, FAKE, None, None, 1.0, FAKE, None, None) == lsh.LSH_ERR_INVALID
    assert f(128, 128, 64, FAKE, FAKE, None, None, 1.0, None, None, None) == lsh.LSH_ERR_INVALID
    assert f(-1, 128, 64, FAKE, FAKE, None, None, 1.0, FAKE, None, None) == lsh.LSH_ERR_INVALID
    assert f(1 << 30, 4096, 64, FAKE, FAKE, None, None, 1.0, FAKE, None, None) == lsh.LSH_ERR_UNSUPPORTED
