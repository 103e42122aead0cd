"""The seeded input generators: determinism, shapes and bf16 rounding."""
import numpy as np
import torch

from paper_2001_04451_amd import workloads as W


def test_bf16_rounding_matches_torch():
    rng = np.random.Generator(np.random.PCG64(0))
    x = np.concatenate([rng.standard_normal(100000).astype(np.float32),
                        np.array([0.0, -0.0, 1.0, 1.00390625, 1.01171875, 3.4e38, -1e-40],
                                 np.float32)])
    ours = W.f32_to_bf16_bits(x)
    theirs = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, theirs)
    back = W.bf16_bits_to_f32(ours)
    assert np.array_equal(back, torch.from_numpy(x).to(torch.bfloat16).float().numpy())


def test_small_workloads_deterministic():
    for name in ("tiny_f32_L1024", "mixture_bf16_L4096"):
        w = W.WORKLOADS[name]
        a, b = W.make_inputs(w), W.make_inputs(w)
        for k in a:
            assert np.array_equal(a[k], b[k])
        assert a["R"].shape == (w.n_rounds, w.d, w.n_buckets // 2)
        assert a["q"].shape == (w.B, w.H, w.L, w.d)
        assert a["q"].dtype == (np.float32 if w.dtype == "f32" else np.uint16)


def test_mixture_is_clustered():
    w = W.WORKLOADS["mixture_bf16_L4096"].scaled(B=1, H=1)
    q = W.as_f64(W.make_inputs(w)["q"], w.dtype)[0, 0]
    # within-component spread is sigma per coordinate; the mixture has at most K
    # distinct centres, so nearest-neighbour distances are far below iid ones
    d2 = ((q[:200, None, :] - q[None, :, :]) ** 2).sum(-1)
    np.fill_diagonal(d2[:, :200], np.inf)
    nn = np.sqrt(d2.min(1))
    assert np.median(nn) < 0.6 * np.sqrt(2 * w.d) * w.sigma * 1.5


def test_all_workloads_declared():
    assert set(W.WORKLOADS) == {"tiny_f32_L1024", "mixture_bf16_L4096", "causal_bf16_L16384",
                                "long_bf16_L65536", "fwdbwd_bf16_L32768"}
    for w in W.WORKLOADS.values():
        assert w.L % w.chunk == 0 and w.n_buckets % 2 == 0
    assert W.WORKLOADS[W.HEADLINE].L == 65536 and W.WORKLOADS[W.HEADLINE].n_rounds == 8
