"""Every output of every entry point is written in full and nothing outside it
is touched.  Each output and each workspace sits inside a larger buffer: the
output region is filled with a value the call cannot produce (NaN for
floating point, 0xFF bytes for exponents, a sentinel for indices) and 4 KiB
guard bands on both sides hold a canary pattern.  After the call (through
the C ABI) every output element must differ from the fill and every guard
byte must be intact.  Cases cover the forward stage by stage, the whole
forward, the backward, the dense baseline and the allocation-free sort, with
partial last chunks and ragged sort tiles."""
import ctypes

import numpy as np
import pytest
import torch

from paper_2001_04451_amd import lsh
from paper_2001_04451_amd import workloads as W

from gpu_common import log, to_device

pytestmark = pytest.mark.gpu

GUARD = 4096  # bytes on each side
CANARY = 0xA5


class Guarded:
    """A device tensor of `shape`/`dtype` inside a buffer with guard bands."""

    def __init__(self, shape, dtype, fill_byte, device):
        self.shape, self.dtype = tuple(shape), dtype
        n = int(np.prod(shape)) * torch.tensor([], dtype=dtype).element_size()
        self.nbytes = n
        self.buf = torch.full((GUARD + n + GUARD,), CANARY, dtype=torch.uint8, device=device)
        self.buf[GUARD:GUARD + n] = fill_byte
        self.t = self.buf[GUARD:GUARD + n].view(dtype).view(self.shape)

    def ptr(self):
        return self.t.data_ptr()

    def check(self, name, unwritten):
        torch.cuda.synchronize()
        b = self.buf.cpu().numpy()
        assert (b[:GUARD] == CANARY).all(), f"{name}: guard band before the buffer overwritten"
        assert (b[GUARD + self.nbytes:] == CANARY).all(), f"{name}: guard band after the buffer overwritten"
        bad = unwritten(self.t)
        assert not bool(bad.any()), f"{name}: {int(bad.sum())} elements left unwritten"


def nan_left(t):
    return torch.isnan(t.float())


def byte_left(t):
    return t == 0xFF


def int_left(t):
    return t == -1  # the 0xFF fill of an int32 buffer


@pytest.fixture(scope="module")
def gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    lsh.lib()
    return torch.device("cuda:0")


def _stream():
    return torch.cuda.current_stream().cuda_stream


def _ws(cfg, dtype, op, dev):
    n = max(256, lsh.workspace_bytes(cfg, dtype, op))
    g = Guarded((n,), torch.uint8, 0x3C, dev)  # the workspace's contents are free
    return g, n


def _check_ws(g, name):
    torch.cuda.synchronize()
    b = g.buf.cpu().numpy()
    assert (b[:GUARD] == CANARY).all() and (b[GUARD + g.nbytes:] == CANARY).all(), \
        f"{name}: workspace guard band overwritten"


@pytest.mark.parametrize("dtype,L,causal", [("bf16", 4160, True), ("bf16", 1000, False),
                                            ("f32", 4000, True), ("f32", 130, False)])
def test_forward_stages_write_exactly_their_outputs(gpu, dtype, L, causal):
    """Hash, sort, chunked attention and combine, each through the C ABI, with
    L not a multiple of the chunk (64) nor of the sort tile (4096)."""
    w = W.WORKLOADS["mixture_bf16_L4096"].scaled(B=1, H=2, L=L, n_rounds=3, dtype=dtype,
                                                 causal=causal)
    x = W.make_inputs(w)
    cfg = lsh.Config.of(w)
    c = cfg.c()
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    code = lsh.LSH_BF16 if dtype == "bf16" else lsh.LSH_F32
    q, v, R = to_device(x["q"], dtype), to_device(x["v"], dtype), to_device(x["R"], "f32")
    B, H, nr, nb, d = w.B, w.H, w.n_rounds, w.n_buckets, w.d
    Lb = lsh.lib()
    log("guards forward", dtype, L, causal)

    buckets = Guarded((B, H, L, nr), torch.int32, 0xFF, gpu)
    ws, n = _ws(cfg, tdt, lsh.LSH_OP_HASH, gpu)
    assert Lb.lsh_hash(ctypes.byref(c), code, q.data_ptr(), R.data_ptr(), buckets.ptr(), ws.t.data_ptr(),
                       n, _stream()) == 0
    buckets.check("buckets", int_left)
    _check_ws(ws, "hash")

    perm = Guarded((B, H, nr, L), torch.int32, 0xFF, gpu)
    undo = Guarded((B, H, nr, L), torch.int32, 0xFF, gpu)
    bstart = Guarded((B, H, nr, nb + 1), torch.int32, 0xFF, gpu)
    ws, n = _ws(cfg, tdt, lsh.LSH_OP_SORT, gpu)
    assert Lb.lsh_sort_permute(ctypes.byref(c), buckets.ptr(), perm.ptr(), undo.ptr(), bstart.ptr(),
                               ws.t.data_ptr(), n, _stream()) == 0
    for name, g in (("perm", perm), ("undo", undo), ("bucket_start", bstart)):
        g.check(name, int_left)
    _check_ws(ws, "sort")

    o_r = Guarded((B, H, nr, L, d), lsh.rounds_dtype(tdt), 0xFF, gpu)
    o_e = Guarded((B, H, nr, L), torch.uint8, 0xFF, gpu) if dtype == "bf16" else None
    lse_r = Guarded((B, H, nr, L), torch.float32, 0xFF, gpu)
    ws, n = _ws(cfg, tdt, lsh.LSH_OP_ATTN_FWD, gpu)
    assert Lb.lsh_chunk_attn_fwd(ctypes.byref(c), code, q.data_ptr(), v.data_ptr(), buckets.ptr(),
                                 perm.ptr(), undo.ptr(), bstart.ptr(), o_r.ptr(),
                                 o_e.ptr() if o_e else None, lse_r.ptr(), ws.t.data_ptr(), n,
                                 _stream()) == 0
    o_r.check("o_rounds", nan_left)
    if o_e:
        o_e.check("o_exp", byte_left)
    lse_r.check("lse_rounds", nan_left)
    _check_ws(ws, "attention")

    out = Guarded((B, H, L, d), tdt, 0xFF, gpu)
    lse = Guarded((B, H, L), torch.float32, 0xFF, gpu)
    assert Lb.lsh_combine_rounds(ctypes.byref(c), code, o_r.ptr(), o_e.ptr() if o_e else None,
                                 lse_r.ptr(), undo.ptr(), out.ptr(), lse.ptr(), _stream()) == 0
    out.check("out", nan_left)
    lse.check("lse_total", nan_left)


@pytest.mark.parametrize("L,causal", [(4160, True), (1000, False), (64, True)])
def test_whole_forward_and_backward_write_exactly_their_outputs(gpu, L, causal):
    w = W.WORKLOADS["fwdbwd_bf16_L32768"].scaled(B=1, H=2, L=L, n_buckets=64, causal=causal)
    x = W.make_inputs(w, with_dout=True)
    cfg = lsh.Config.of(w)
    c = cfg.c()
    tdt = torch.bfloat16
    q, v, R = to_device(x["q"], "bf16"), to_device(x["v"], "bf16"), to_device(x["R"], "f32")
    dout = to_device(x["dout"], "bf16")
    B, H, nr, nb, d = w.B, w.H, w.n_rounds, w.n_buckets, w.d
    Lb = lsh.lib()
    log("guards forward+backward", L, causal)
    out = Guarded((B, H, L, d), tdt, 0xFF, gpu)
    lse = Guarded((B, H, L), torch.float32, 0xFF, gpu)
    buckets = Guarded((B, H, L, nr), torch.int32, 0xFF, gpu)
    perm = Guarded((B, H, nr, L), torch.int32, 0xFF, gpu)
    undo = Guarded((B, H, nr, L), torch.int32, 0xFF, gpu)
    bstart = Guarded((B, H, nr, nb + 1), torch.int32, 0xFF, gpu)
    ws, n = _ws(cfg, tdt, lsh.LSH_OP_FORWARD, gpu)
    assert Lb.lsh_attention_fwd(ctypes.byref(c), lsh.LSH_BF16, q.data_ptr(), v.data_ptr(), R.data_ptr(),
                                out.ptr(), lse.ptr(), buckets.ptr(), perm.ptr(), undo.ptr(),
                                bstart.ptr(), ws.t.data_ptr(), n, _stream()) == 0
    out.check("out", nan_left)
    lse.check("lse_total", nan_left)
    for name, g in (("buckets", buckets), ("perm", perm), ("undo", undo), ("bucket_start", bstart)):
        g.check(name, int_left)
    _check_ws(ws, "forward")

    dq = Guarded((B, H, L, d), torch.float32, 0xFF, gpu)
    dv = Guarded((B, H, L, d), torch.float32, 0xFF, gpu)
    ws, n = _ws(cfg, tdt, lsh.LSH_OP_ATTN_BWD, gpu)
    assert Lb.lsh_chunk_attn_bwd(ctypes.byref(c), lsh.LSH_BF16, q.data_ptr(), v.data_ptr(), out.ptr(),
                                 dout.data_ptr(), lse.ptr(), buckets.ptr(), perm.ptr(), undo.ptr(),
                                 bstart.ptr(), dq.ptr(), dv.ptr(), ws.t.data_ptr(), n, _stream()) == 0
    dq.check("dq", nan_left)
    dv.check("dv", nan_left)
    _check_ws(ws, "backward")

    # the allocation-free sort on the same ids
    perm2 = Guarded((B, H, nr, L), torch.int32, 0xFF, gpu)
    undo2 = Guarded((B, H, nr, L), torch.int32, 0xFF, gpu)
    bstart2 = Guarded((B, H, nr, nb + 1), torch.int32, 0xFF, gpu)
    assert Lb.lsh_sort_permute_static(ctypes.byref(c), buckets.ptr(), perm2.ptr(), undo2.ptr(),
                                      bstart2.ptr(), _stream()) == 0
    for name, g in (("static perm", perm2), ("static undo", undo2), ("static bucket_start", bstart2)):
        g.check(name, int_left)


def test_dense_writes_exactly_its_outputs(gpu):
    w = W.WORKLOADS["mixture_bf16_L4096"].scaled(B=1, H=2, L=300, causal=True)
    x = W.make_inputs(w)
    cfg = lsh.Config(B=w.B, H=w.H, L=w.L, n_buckets=2, n_rounds=1, causal=True)
    c = cfg.c()
    q, v = to_device(x["q"], "bf16"), to_device(x["v"], "bf16")
    log("guards dense")
    out = Guarded((w.B, w.H, w.L, w.d), torch.bfloat16, 0xFF, gpu)
    lse = Guarded((w.B, w.H, w.L), torch.float32, 0xFF, gpu)
    ws, n = _ws(cfg, torch.bfloat16, lsh.LSH_OP_DENSE_FWD, gpu)
    assert lsh.lib().lsh_dense_attn_fwd(ctypes.byref(c), lsh.LSH_BF16, q.data_ptr(), v.data_ptr(),
                                        out.ptr(), lse.ptr(), ws.t.data_ptr(), n, _stream()) == 0
    out.check("dense out", nan_left)
    lse.check("dense lse", nan_left)
    _check_ws(ws, "dense")
