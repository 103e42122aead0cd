"""lsh_sort_permute_static (no workspace argument, a fixed scratch array inside
the library) against lsh_sort_permute (caller's workspace), through the C ABI,
bit for bit: two calls in a row, the second on a smaller input, so the second
call runs on scratch the first one left behind."""
import ctypes

import numpy as np
import pytest
import torch

from paper_2001_04451_amd import lsh

pytestmark = pytest.mark.gpu


def _ids(B, H, L, n_r, n_b, seed):
    rng = np.random.Generator(np.random.PCG64(seed))
    return torch.from_numpy(rng.integers(0, n_b, size=(B, H, L, n_r)).astype(np.int32)).cuda()


def _static_sort(cfg, buckets):
    dev = buckets.device
    perm = torch.full((cfg.B, cfg.H, cfg.n_rounds, cfg.L), -7, dtype=torch.int32, device=dev)
    undo = torch.full_like(perm, -7)
    bstart = torch.full((cfg.B, cfg.H, cfg.n_rounds, cfg.n_buckets + 1), -7, dtype=torch.int32,
                        device=dev)
    stream = torch.cuda.current_stream(dev).cuda_stream
    print(f"[gpu-case] sort static B={cfg.B} H={cfg.H} L={cfg.L} n_r={cfg.n_rounds} "
          f"n_b={cfg.n_buckets}", flush=True)
    rc = lsh.lib().lsh_sort_permute_static(ctypes.byref(cfg.c()), buckets.data_ptr(),
                                           perm.data_ptr(), undo.data_ptr(), bstart.data_ptr(),
                                           stream)
    assert rc == lsh.LSH_OK, lsh.lib().lsh_status_string(rc)
    return perm, undo, bstart


def test_static_sort_matches_workspace_sort():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    lsh.lib()
    # the benchmark's shape first (8 MiB of counts), then a smaller, ragged one
    for (B, H, L, n_r, n_b, seed) in [(1, 16, 65536, 8, 1024, 5), (2, 3, 5000, 3, 256, 6)]:
        cfg = lsh.Config(B=B, H=H, L=L, n_buckets=n_b, n_rounds=n_r)
        buckets = _ids(B, H, L, n_r, n_b, seed)
        p_s, u_s, b_s = _static_sort(cfg, buckets)
        p_w, u_w, b_w = lsh.lsh_sort_permute(cfg, buckets)
        torch.cuda.synchronize()
        assert torch.equal(p_s, p_w)
        assert torch.equal(u_s, u_w)
        assert torch.equal(b_s, b_w)


def test_static_sort_refuses_oversized_counts():
    """Counts beyond the fixed 16 MiB scratch: refused before any HIP call."""
    cfg = lsh.Config(B=8, H=16, L=65536, n_buckets=1024, n_rounds=8)  # 64 MiB of counts
    fake = ctypes.c_void_p(0x1000)
    rc = lsh.lib().lsh_sort_permute_static(ctypes.byref(cfg.c()), fake, fake, fake, fake, None)
    assert rc == lsh.LSH_ERR_UNSUPPORTED
