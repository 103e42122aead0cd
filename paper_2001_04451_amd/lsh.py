"""Thin Python binding of liblsh (the C ABI in include/lsh.h).

Two layers:
  * ``lib()`` exposes the raw C entry points; they take an ``LshConfig``,
    raw device pointers (ints), sizes and a stream handle, and return the
    status code unchanged.
  * The module functions of the same names (``lsh_hash``,
    ``lsh_sort_permute``, ``lsh_chunk_attn_fwd``, ...) marshal torch tensors: they check shapes and dtypes, allocate outputs and
    workspace with torch, call the C entry point on torch's current stream
    and raise ``LshError`` on a non-zero status.  All arithmetic happens in
    the HIP kernels behind the C ABI.

Nothing here falls back to another implementation: if liblsh.so is missing
or fails to load, importing a compute function raises.
"""
from __future__ import annotations

import ctypes
import math
import os
from dataclasses import dataclass

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "liblsh.so")

LSH_OK, LSH_ERR_INVALID, LSH_ERR_UNSUPPORTED, LSH_ERR_HIP = 0, -1, -2, -3
LSH_F32, LSH_BF16 = 0, 1
(LSH_OP_HASH, LSH_OP_SORT, LSH_OP_ATTN_FWD, LSH_OP_COMBINE, LSH_OP_ATTN_BWD,
 LSH_OP_FORWARD, LSH_OP_DENSE_FWD) = range(7)

# Every symbol include/lsh.h declares.
EXPORTED = ("lsh_status_string", "lsh_workspace_bytes", "lsh_hash", "lsh_sort_permute",
            "lsh_sort_permute_static",
            "lsh_gather_rows", "lsh_chunk_attn_fwd", "lsh_combine_rounds", "lsh_attention_fwd",
            "lsh_chunk_attn_bwd", "lsh_dense_attn_fwd",
            # include/lsh_block.h
            "lsh_block_workspace_bytes", "lsh_rev_attention", "lsh_rev_feed_forward",
            "lsh_rev_block_fwd", "lsh_rev_block_inv", "lsh_linear_bf16")
LSH_BLOCK_OP_ATTN, LSH_BLOCK_OP_FF, LSH_BLOCK_OP_BLOCK = 0, 1, 2


class LshConfig(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int32), ("H", ctypes.c_int32), ("L", ctypes.c_int32),
                ("d", ctypes.c_int32), ("n_buckets", ctypes.c_int32),
                ("n_rounds", ctypes.c_int32), ("chunk", ctypes.c_int32),
                ("causal", ctypes.c_int32), ("scale", ctypes.c_float),
                ("self_mask", ctypes.c_float), ("chunks_after", ctypes.c_int32),
                ("attend_across", ctypes.c_int32), ("r_per_head", ctypes.c_int32)]


class BlockConfigC(ctypes.Structure):
    _fields_ = [("attn", LshConfig), ("d_ff", ctypes.c_int32), ("ff_chunk", ctypes.c_int32),
                ("ln_eps", ctypes.c_float)]


class BlockWeightsC(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in ("ln1_g", "ln1_b", "w_qk", "w_v", "w_o", "R", "ln2_g",
                                               "ln2_b", "w1", "b1", "w2", "b2")]


class LshError(RuntimeError):
    def __init__(self, call: str, status: int):
        msg = _lib.lsh_status_string(status).decode() if _lib is not None else str(status)
        super().__init__(f"{call} failed: {msg} ({status})")
        self.status = status


_lib = None
_P = ctypes.c_void_p
_CFG = ctypes.POINTER(LshConfig)
_BCFG = ctypes.POINTER(BlockConfigC)
_BW = ctypes.POINTER(BlockWeightsC)
_SZ = ctypes.c_size_t
_I = ctypes.c_int


def lib() -> ctypes.CDLL:
    """Load liblsh.so (built by paper_2001_04451_amd.build); raise if absent."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is not built; run `python -m paper_2001_04451_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        L.lsh_status_string.argtypes = [_I]
        L.lsh_status_string.restype = ctypes.c_char_p
        L.lsh_workspace_bytes.argtypes = [_CFG, _I, _I]
        L.lsh_workspace_bytes.restype = _SZ
        sigs = {
            "lsh_hash": [_CFG, _I, _P, _P, _P, _P, _SZ, _P],
            "lsh_sort_permute": [_CFG, _P, _P, _P, _P, _P, _SZ, _P],
            "lsh_sort_permute_static": [_CFG, _P, _P, _P, _P, _P],
            "lsh_gather_rows": [_CFG, _I, _P, _P, _P, _P],
            "lsh_chunk_attn_fwd": [_CFG, _I, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _SZ, _P],
            "lsh_combine_rounds": [_CFG, _I, _P, _P, _P, _P, _P, _P, _P],
            "lsh_attention_fwd": [_CFG, _I, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _SZ, _P],
            "lsh_chunk_attn_bwd": [_CFG, _I, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _SZ,
                                   _P],
            "lsh_dense_attn_fwd": [_CFG, _I, _P, _P, _P, _P, _P, _SZ, _P],
            "lsh_rev_attention": [_BCFG, _BW, _P, _P, _P, ctypes.c_float, _P, _SZ, _P],
            "lsh_rev_feed_forward": [_BCFG, _BW, _P, _P, _P, ctypes.c_float, _P, _SZ, _P],
            "lsh_rev_block_fwd": [_BCFG, _BW, _P, _P, _P, _P, _P, _SZ, _P],
            "lsh_rev_block_inv": [_BCFG, _BW, _P, _P, _P, _P, _P, _SZ, _P],
            "lsh_linear_bf16": [ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, _P, _P, _P, _P,
                                ctypes.c_float, _P, _P, _P],
        }
        L.lsh_block_workspace_bytes.argtypes = [_BCFG, _I]
        L.lsh_block_workspace_bytes.restype = _SZ
        for name, args in sigs.items():
            fn = getattr(L, name)
            fn.argtypes = args
            fn.restype = _I
        _lib = L
    return _lib


# --------------------------------------------------------------------------
# configuration
# --------------------------------------------------------------------------
@dataclass(frozen=True)
class Config:
    B: int
    H: int
    L: int
    n_buckets: int
    n_rounds: int
    chunk: int = 64
    causal: bool = False
    d: int = 64
    scale: float | None = None
    self_mask: float = 1e5
    chunks_after: int = 0
    attend_across: bool = False
    r_per_head: bool = False

    def c(self) -> LshConfig:
        scale = 1.0 / math.sqrt(self.d) if self.scale is None else self.scale
        return LshConfig(self.B, self.H, self.L, self.d, self.n_buckets, self.n_rounds, self.chunk,
                         int(bool(self.causal)), scale, self.self_mask, int(self.chunks_after),
                         int(bool(self.attend_across)), int(bool(self.r_per_head)))

    def r_shape(self) -> tuple:
        """Shape of R: one set per round, or per head and round with r_per_head."""
        base = (self.n_rounds, self.d, self.n_buckets // 2)
        return (self.H,) + base if self.r_per_head else base

    @staticmethod
    def of(w, **kw) -> "Config":
        """From a workloads.Workload (keyword arguments override fields)."""
        c = dict(B=w.B, H=w.H, L=w.L, n_buckets=w.n_buckets, n_rounds=w.n_rounds, chunk=w.chunk,
                 causal=w.causal, d=w.d)
        c.update(kw)
        return Config(**c)


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return LSH_F32
    if t.dtype == torch.bfloat16:
        return LSH_BF16
    raise TypeError(f"unsupported dtype {t.dtype}; use float32 or bfloat16")


def _ptr(t: torch.Tensor | None) -> int | None:
    return None if t is None else t.data_ptr()


def _stream(device: torch.device) -> int:
    return torch.cuda.current_stream(device).cuda_stream


def _check(call: str, status: int) -> None:
    if status != LSH_OK:
        raise LshError(call, status)


def _need(t: torch.Tensor, shape, dtype=None, name="tensor") -> None:
    if not t.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} has dtype {t.dtype}, expected {dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def workspace_bytes(cfg: Config, dtype: torch.dtype, op: int) -> int:
    code = LSH_BF16 if dtype == torch.bfloat16 else LSH_F32
    return int(lib().lsh_workspace_bytes(ctypes.byref(cfg.c()), code, op))


def _workspace(cfg: Config, dtype: torch.dtype, op: int, device) -> torch.Tensor:
    n = workspace_bytes(cfg, dtype, op)
    return torch.empty(max(n, 256), dtype=torch.uint8, device=device)


# --------------------------------------------------------------------------
# torch-level calls, one per C entry point
# --------------------------------------------------------------------------
def lsh_hash(cfg: Config, q: torch.Tensor, R: torch.Tensor, buckets: torch.Tensor | None = None,
         workspace: torch.Tensor | None = None) -> torch.Tensor:
    """Bucket ids [B,H,L,n_rounds] int32 (lsh_hash)."""
    _need(q, (cfg.B, cfg.H, cfg.L, cfg.d), name="q")
    _need(R, cfg.r_shape(), torch.float32, "R")
    if buckets is None:
        buckets = torch.empty((cfg.B, cfg.H, cfg.L, cfg.n_rounds), dtype=torch.int32, device=q.device)
    if workspace is None:
        workspace = _workspace(cfg, q.dtype, LSH_OP_HASH, q.device)
    _check("lsh_hash", lib().lsh_hash(ctypes.byref(cfg.c()), _dtype_code(q), _ptr(q), _ptr(R),
                                      _ptr(buckets), _ptr(workspace), workspace.numel(),
                                      _stream(q.device)))
    return buckets


def lsh_sort_permute(cfg: Config, buckets: torch.Tensor, workspace: torch.Tensor | None = None,
                     perm=None, undo=None, bstart=None):
    """perm, undo [B,H,n_r,L] and bucket_start [B,H,n_r,n_b+1] (lsh_sort_permute)."""
    _need(buckets, (cfg.B, cfg.H, cfg.L, cfg.n_rounds), torch.int32, "buckets")
    dev = buckets.device
    if perm is None:
        perm = torch.empty((cfg.B, cfg.H, cfg.n_rounds, cfg.L), dtype=torch.int32, device=dev)
    if undo is None:
        undo = torch.empty_like(perm)
    if bstart is None:
        bstart = torch.empty((cfg.B, cfg.H, cfg.n_rounds, cfg.n_buckets + 1), dtype=torch.int32,
                             device=dev)
    _need(perm, (cfg.B, cfg.H, cfg.n_rounds, cfg.L), torch.int32, "perm")
    _need(undo, (cfg.B, cfg.H, cfg.n_rounds, cfg.L), torch.int32, "undo")
    _need(bstart, (cfg.B, cfg.H, cfg.n_rounds, cfg.n_buckets + 1), torch.int32, "bucket_start")
    if workspace is None:
        workspace = _workspace(cfg, torch.float32, LSH_OP_SORT, dev)
    _check("lsh_sort_permute",
           lib().lsh_sort_permute(ctypes.byref(cfg.c()), _ptr(buckets), _ptr(perm), _ptr(undo),
                                  _ptr(bstart), _ptr(workspace), workspace.numel(), _stream(dev)))
    return perm, undo, bstart


def lsh_gather_rows(cfg: Config, src: torch.Tensor, perm: torch.Tensor) -> torch.Tensor:
    """Rows of src in sorted order [B,H,n_r,L,d] (lsh_gather_rows)."""
    _need(src, (cfg.B, cfg.H, cfg.L, cfg.d), name="src")
    _need(perm, (cfg.B, cfg.H, cfg.n_rounds, cfg.L), torch.int32, "perm")
    dst = torch.empty((cfg.B, cfg.H, cfg.n_rounds, cfg.L, cfg.d), dtype=src.dtype, device=src.device)
    _check("lsh_gather_rows", lib().lsh_gather_rows(ctypes.byref(cfg.c()), _dtype_code(src),
                                                    _ptr(src), _ptr(perm), _ptr(dst),
                                                    _stream(src.device)))
    return dst


def rounds_dtype(dtype: torch.dtype) -> torch.dtype:
    """Element type of o_rounds for a call in `dtype`: fp32 for fp32 calls, fp16
    (each row scaled by 2^-o_exp) for bf16 calls."""
    return torch.float32 if dtype == torch.float32 else torch.float16


def lsh_chunk_attn_fwd(cfg: Config, q, v, buckets, perm, bstart, o_rounds=None, o_exp=None,
                       lse_rounds=None, workspace=None, undo=None):
    """Per-round outputs in sorted order (lsh_chunk_attn_fwd): o_rounds [B,H,n_r,L,d]
    (fp32 for fp32 q; fp16 scaled by 2^-o_exp for bf16 q), o_exp [B,H,n_r,L] uint8
    (None for fp32 q) and lse_rounds [B,H,n_r,L] fp32."""
    _need(q, (cfg.B, cfg.H, cfg.L, cfg.d), name="q")
    _need(v, (cfg.B, cfg.H, cfg.L, cfg.d), q.dtype, "v")
    _need(perm, (cfg.B, cfg.H, cfg.n_rounds, cfg.L), torch.int32, "perm")
    _need(bstart, (cfg.B, cfg.H, cfg.n_rounds, cfg.n_buckets + 1), torch.int32, "bucket_start")
    _need(buckets, (cfg.B, cfg.H, cfg.L, cfg.n_rounds), torch.int32, "buckets")
    if undo is not None:
        _need(undo, (cfg.B, cfg.H, cfg.n_rounds, cfg.L), torch.int32, "undo")
    elif cfg.attend_across:
        raise ValueError("undo is required with attend_across")
    dev = q.device
    rdt = rounds_dtype(q.dtype)
    if o_rounds is None:
        o_rounds = torch.empty((cfg.B, cfg.H, cfg.n_rounds, cfg.L, cfg.d), dtype=rdt,
                               device=dev)
    _need(o_rounds, (cfg.B, cfg.H, cfg.n_rounds, cfg.L, cfg.d), rdt, "o_rounds")
    if q.dtype != torch.float32:
        if o_exp is None:
            o_exp = torch.empty((cfg.B, cfg.H, cfg.n_rounds, cfg.L), dtype=torch.uint8,
                                device=dev)
        _need(o_exp, (cfg.B, cfg.H, cfg.n_rounds, cfg.L), torch.uint8, "o_exp")
    else:
        o_exp = None
    if lse_rounds is None:
        lse_rounds = torch.empty((cfg.B, cfg.H, cfg.n_rounds, cfg.L), dtype=torch.float32,
                                 device=dev)
    _need(lse_rounds, (cfg.B, cfg.H, cfg.n_rounds, cfg.L), torch.float32, "lse_rounds")
    if workspace is None:
        workspace = _workspace(cfg, q.dtype, LSH_OP_ATTN_FWD, dev)
    _check("lsh_chunk_attn_fwd",
           lib().lsh_chunk_attn_fwd(ctypes.byref(cfg.c()), _dtype_code(q), _ptr(q), _ptr(v),
                                    _ptr(buckets), _ptr(perm), _ptr(undo), _ptr(bstart), _ptr(o_rounds),
                                    _ptr(o_exp), _ptr(lse_rounds), _ptr(workspace),
                                    workspace.numel(), _stream(dev)))
    return o_rounds, o_exp, lse_rounds


def lsh_combine_rounds(cfg: Config, o_rounds, o_exp, lse_rounds, undo, out_dtype: torch.dtype,
                       out=None, lse_total=None):
    """Output [B,H,L,d] in out_dtype and lse_total [B,H,L] fp32 (lsh_combine_rounds).
    o_rounds, o_exp and lse_rounds as lsh_chunk_attn_fwd writes them for a call in
    out_dtype."""
    _need(o_rounds, (cfg.B, cfg.H, cfg.n_rounds, cfg.L, cfg.d), rounds_dtype(out_dtype),
          "o_rounds")
    if out_dtype != torch.float32:
        if o_exp is None:
            raise ValueError("o_exp is required for bf16 calls")
        _need(o_exp, (cfg.B, cfg.H, cfg.n_rounds, cfg.L), torch.uint8, "o_exp")
    _need(lse_rounds, (cfg.B, cfg.H, cfg.n_rounds, cfg.L), torch.float32, "lse_rounds")
    _need(undo, (cfg.B, cfg.H, cfg.n_rounds, cfg.L), torch.int32, "undo")
    dev = o_rounds.device
    if out is None:
        out = torch.empty((cfg.B, cfg.H, cfg.L, cfg.d), dtype=out_dtype, device=dev)
    _need(out, (cfg.B, cfg.H, cfg.L, cfg.d), out_dtype, "out")
    if lse_total is None:
        lse_total = torch.empty((cfg.B, cfg.H, cfg.L), dtype=torch.float32, device=dev)
    _check("lsh_combine_rounds",
           lib().lsh_combine_rounds(ctypes.byref(cfg.c()), _dtype_code(out), _ptr(o_rounds),
                                    _ptr(o_exp), _ptr(lse_rounds), _ptr(undo), _ptr(out),
                                    _ptr(lse_total), _stream(dev)))
    return out, lse_total


class ForwardState:
    """Buffers of one forward pass; reusable across calls of the same shape."""

    def __init__(self, cfg: Config, dtype: torch.dtype, device):
        self.cfg = cfg
        B, H, L, nr, nb = cfg.B, cfg.H, cfg.L, cfg.n_rounds, cfg.n_buckets
        self.out = torch.empty((B, H, L, cfg.d), dtype=dtype, device=device)
        self.lse = torch.empty((B, H, L), dtype=torch.float32, device=device)
        self.buckets = torch.empty((B, H, L, nr), dtype=torch.int32, device=device)
        self.perm = torch.empty((B, H, nr, L), dtype=torch.int32, device=device)
        self.undo = torch.empty_like(self.perm)
        self.bstart = torch.empty((B, H, nr, nb + 1), dtype=torch.int32, device=device)
        self.workspace = _workspace(cfg, dtype, LSH_OP_FORWARD, device)


def lsh_attention_fwd(cfg: Config, q, v, R, state: ForwardState | None = None) -> ForwardState:
    """The whole forward (lsh_attention_fwd): hash, sort, chunked attention, combine."""
    _need(q, (cfg.B, cfg.H, cfg.L, cfg.d), name="q")
    _need(v, (cfg.B, cfg.H, cfg.L, cfg.d), q.dtype, "v")
    _need(R, cfg.r_shape(), torch.float32, "R")
    if state is None:
        state = ForwardState(cfg, q.dtype, q.device)
    s = state
    _check("lsh_attention_fwd",
           lib().lsh_attention_fwd(ctypes.byref(cfg.c()), _dtype_code(q), _ptr(q), _ptr(v), _ptr(R),
                                   _ptr(s.out), _ptr(s.lse), _ptr(s.buckets), _ptr(s.perm),
                                   _ptr(s.undo), _ptr(s.bstart), _ptr(s.workspace),
                                   s.workspace.numel(), _stream(q.device)))
    return state


def lsh_chunk_attn_bwd(cfg: Config, q, v, out, dout, lse_total, buckets, perm, undo, bstart,
                   dq=None, dv=None, workspace=None):
    """dq, dv [B,H,L,d] fp32 (lsh_chunk_attn_bwd)."""
    shp = (cfg.B, cfg.H, cfg.L, cfg.d)
    _need(q, shp, name="q")
    for name, t in (("v", v), ("out", out), ("dout", dout)):
        _need(t, shp, q.dtype, name)
    _need(lse_total, (cfg.B, cfg.H, cfg.L), torch.float32, "lse_total")
    _need(buckets, (cfg.B, cfg.H, cfg.L, cfg.n_rounds), torch.int32, "buckets")
    _need(perm, (cfg.B, cfg.H, cfg.n_rounds, cfg.L), torch.int32, "perm")
    _need(undo, (cfg.B, cfg.H, cfg.n_rounds, cfg.L), torch.int32, "undo")
    _need(bstart, (cfg.B, cfg.H, cfg.n_rounds, cfg.n_buckets + 1), torch.int32, "bucket_start")
    dev = q.device
    if dq is None:
        dq = torch.empty(shp, dtype=torch.float32, device=dev)
    if dv is None:
        dv = torch.empty(shp, dtype=torch.float32, device=dev)
    _need(dq, shp, torch.float32, "dq")
    _need(dv, shp, torch.float32, "dv")
    if workspace is None:
        workspace = _workspace(cfg, q.dtype, LSH_OP_ATTN_BWD, dev)
    _check("lsh_chunk_attn_bwd",
           lib().lsh_chunk_attn_bwd(ctypes.byref(cfg.c()), _dtype_code(q), _ptr(q), _ptr(v),
                                    _ptr(out), _ptr(dout), _ptr(lse_total), _ptr(buckets),
                                    _ptr(perm), _ptr(undo), _ptr(bstart), _ptr(dq), _ptr(dv),
                                    _ptr(workspace), workspace.numel(), _stream(dev)))
    return dq, dv


def lsh_dense_attn_fwd(cfg: Config, q, v, out=None, lse=None, workspace=None):
    """Full shared-QK attention (lsh_dense_attn_fwd): out [B,H,L,d] bf16 and
    lse [B,H,L] fp32.  Only the shape, causal flag and scales of cfg are used."""
    _need(q, (cfg.B, cfg.H, cfg.L, cfg.d), torch.bfloat16, "q")
    _need(v, (cfg.B, cfg.H, cfg.L, cfg.d), torch.bfloat16, "v")
    dev = q.device
    if out is None:
        out = torch.empty_like(q)
    _need(out, (cfg.B, cfg.H, cfg.L, cfg.d), torch.bfloat16, "out")
    if lse is None:
        lse = torch.empty((cfg.B, cfg.H, cfg.L), dtype=torch.float32, device=dev)
    if workspace is None:
        workspace = _workspace(cfg, q.dtype, LSH_OP_DENSE_FWD, dev)
    _check("lsh_dense_attn_fwd",
           lib().lsh_dense_attn_fwd(ctypes.byref(cfg.c()), _dtype_code(q), _ptr(q), _ptr(v),
                                    _ptr(out), _ptr(lse), _ptr(workspace), workspace.numel(),
                                    _stream(dev)))
    return out, lse


# --------------------------------------------------------------------------
# the reversible block (include/lsh_block.h)
# --------------------------------------------------------------------------
@dataclass(frozen=True)
class BlockConfig:
    attn: Config
    d_ff: int
    ff_chunk: int = 0
    ln_eps: float = 1e-5

    @property
    def d_model(self) -> int:
        return 64 * self.attn.H

    @property
    def rows(self) -> int:
        return self.attn.B * self.attn.L

    def c(self) -> BlockConfigC:
        return BlockConfigC(self.attn.c(), self.d_ff, self.ff_chunk, self.ln_eps)

    @staticmethod
    def of(w, **kw) -> "BlockConfig":
        """From a workloads.BlockWorkload (keyword arguments override fields)."""
        attn = Config(B=w.B, H=w.H, L=w.L, n_buckets=w.n_buckets, n_rounds=w.n_rounds, chunk=w.chunk,
                      causal=w.causal)
        c = dict(attn=attn, d_ff=w.d_ff, ff_chunk=w.ff_chunk, ln_eps=w.ln_eps)
        c.update(kw)
        return BlockConfig(**c)


_WEIGHT_NAMES = ("ln1_g", "ln1_b", "w_qk", "w_v", "w_o", "R", "ln2_g", "ln2_b", "w1", "b1", "w2", "b2")


class BlockWeights:
    """Device tensors of the block's weights (bf16 matrices, fp32 vectors and R)."""

    def __init__(self, **tensors):
        for n in _WEIGHT_NAMES:
            setattr(self, n, tensors[n])

    def c(self) -> BlockWeightsC:
        return BlockWeightsC(*[_ptr(getattr(self, n)) for n in _WEIGHT_NAMES])


def block_workspace_bytes(cfg: BlockConfig, op: int) -> int:
    return int(lib().lsh_block_workspace_bytes(ctypes.byref(cfg.c()), op))


def _block_ws(cfg: BlockConfig, op: int, device) -> torch.Tensor:
    return torch.empty(max(block_workspace_bytes(cfg, op), 256), dtype=torch.uint8, device=device)


def _rows(cfg: BlockConfig, t: torch.Tensor, name: str) -> None:
    _need(t, (cfg.attn.B, cfg.attn.L, cfg.d_model), torch.float32, name)


def rev_attention(cfg: BlockConfig, w: BlockWeights, x, resid=None, sign: float = 1.0, out=None,
                  workspace=None):
    """out = resid + sign * F(x) (lsh_rev_attention)."""
    _rows(cfg, x, "x")
    if resid is not None:
        _rows(cfg, resid, "resid")
    out = torch.empty_like(x) if out is None else out
    _rows(cfg, out, "out")
    ws = _block_ws(cfg, LSH_BLOCK_OP_ATTN, x.device) if workspace is None else workspace
    _check("lsh_rev_attention",
           lib().lsh_rev_attention(ctypes.byref(cfg.c()), ctypes.byref(w.c()), _ptr(x), _ptr(resid), _ptr(out),
                                   sign, _ptr(ws), ws.numel(), _stream(x.device)))
    return out


def rev_feed_forward(cfg: BlockConfig, w: BlockWeights, x, resid=None, sign: float = 1.0, out=None,
                     workspace=None):
    """out = resid + sign * G(x), chunked (lsh_rev_feed_forward)."""
    _rows(cfg, x, "x")
    if resid is not None:
        _rows(cfg, resid, "resid")
    out = torch.empty_like(x) if out is None else out
    _rows(cfg, out, "out")
    ws = _block_ws(cfg, LSH_BLOCK_OP_FF, x.device) if workspace is None else workspace
    _check("lsh_rev_feed_forward",
           lib().lsh_rev_feed_forward(ctypes.byref(cfg.c()), ctypes.byref(w.c()), _ptr(x), _ptr(resid),
                                      _ptr(out), sign, _ptr(ws), ws.numel(), _stream(x.device)))
    return out


def rev_block_fwd(cfg: BlockConfig, w: BlockWeights, x1, x2, y1=None, y2=None, workspace=None):
    """(y1, y2) = (x1 + F(x2), x2 + G(y1)) (lsh_rev_block_fwd)."""
    for t, n in ((x1, "x1"), (x2, "x2")):
        _rows(cfg, t, n)
    y1 = torch.empty_like(x1) if y1 is None else y1
    y2 = torch.empty_like(x2) if y2 is None else y2
    ws = _block_ws(cfg, LSH_BLOCK_OP_BLOCK, x1.device) if workspace is None else workspace
    _check("lsh_rev_block_fwd",
           lib().lsh_rev_block_fwd(ctypes.byref(cfg.c()), ctypes.byref(w.c()), _ptr(x1), _ptr(x2), _ptr(y1),
                                   _ptr(y2), _ptr(ws), ws.numel(), _stream(x1.device)))
    return y1, y2


def rev_block_inv(cfg: BlockConfig, w: BlockWeights, y1, y2, x1=None, x2=None, workspace=None):
    """(x1, x2) = (y1 - F(x2), y2 - G(y1)) (lsh_rev_block_inv)."""
    for t, n in ((y1, "y1"), (y2, "y2")):
        _rows(cfg, t, n)
    x1 = torch.empty_like(y1) if x1 is None else x1
    x2 = torch.empty_like(y2) if x2 is None else x2
    ws = _block_ws(cfg, LSH_BLOCK_OP_BLOCK, y1.device) if workspace is None else workspace
    _check("lsh_rev_block_inv",
           lib().lsh_rev_block_inv(ctypes.byref(cfg.c()), ctypes.byref(w.c()), _ptr(y1), _ptr(y2), _ptr(x1),
                                   _ptr(x2), _ptr(ws), ws.numel(), _stream(y1.device)))
    return x1, x2


def linear_bf16(a: torch.Tensor, w: torch.Tensor, bias=None, resid=None, sign: float = 1.0,
                relu_bf16: bool = False) -> torch.Tensor:
    """The block's product (lsh_linear_bf16): resid + sign (a w^T + bias) in
    fp32, or bf16(relu(a w^T + bias)) with relu_bf16."""
    M, K = a.shape
    N = w.shape[0]
    _need(a, (M, K), torch.bfloat16, "a")
    _need(w, (N, K), torch.bfloat16, "w")
    if relu_bf16:
        out = torch.empty((M, N), dtype=torch.bfloat16, device=a.device)
        args = (None, _ptr(out))
    else:
        out = torch.empty((M, N), dtype=torch.float32, device=a.device)
        args = (_ptr(out), None)
    _check("lsh_linear_bf16",
           lib().lsh_linear_bf16(M, N, K, _ptr(a), _ptr(w), _ptr(bias), _ptr(resid), sign, *args,
                                 _stream(a.device)))
    return out
