"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer, on the
CPU: the oracle (built with gcc and the sanitizers) runs every routine on
small cases, and the C ABI's argument validation (lsh_api.cpp built with the
host-side sanitizers and linked with the kernel objects of the normal build)
runs its refusal paths.  Each runs in a child process with the sanitizer
runtime preloaded; any report fails the test."""
import glob
import os
import shutil
import subprocess
import sys
import textwrap

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2001_04451_amd")


def _run(code: str, env_extra: dict) -> subprocess.CompletedProcess:
    env = dict(os.environ)
    env.update(env_extra)
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=1"
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1"
    env["PYTHONPATH"] = ROOT
    return subprocess.run([sys.executable, "-c", textwrap.dedent(code)], env=env,
                          capture_output=True, text=True, timeout=600)


def test_oracle_under_sanitizers(tmp_path):
    lib = str(tmp_path / "liblsh_oracle_san.so")
    subprocess.check_call(["gcc", "-O1", "-g", "-std=c11", "-fopenmp", "-fPIC", "-shared",
                           "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
                           "-fno-omit-frame-pointer", os.path.join(ROOT, "oracle", "lsh_oracle.c"),
                           "-o", lib, "-lm"])
    asan = subprocess.check_output(["gcc", "-print-file-name=libasan.so"], text=True).strip()
    ubsan = subprocess.check_output(["gcc", "-print-file-name=libubsan.so"], text=True).strip()
    res = _run("""
        import numpy as np
        import oracle
        rng = np.random.default_rng(0)
        for (L, m, nb, nr, causal, after, across) in [(100, 16, 8, 3, True, 0, False),
                                                        (203, 32, 4, 2, False, 1, False),
                                                        (96, 16, 8, 3, True, 1, True),
                                                        (64, 64, 2, 1, False, 0, True)]:
            q = rng.standard_normal((2, 2, L, 16))
            v = rng.standard_normal((2, 2, L, 16))
            dO = rng.standard_normal((2, 2, L, 16))
            R = rng.standard_normal((2, nr, 16, nb // 2))  # one R per head
            ref = oracle.lsh_attention_fwd(q, v, R, m, causal, after=after, across=across)
            oracle.lsh_chunk_attn_bwd(q, v, ref["out"], dO, ref["lse"], ref["buckets"], ref["perm"],
                                      m, causal, after=after, across=across)
            oracle.dense_attn_fwd(q, v, causal)
            oracle.dense_attn_fwd(q, v, causal, rows=[0, 5, L + 3])
        print("ok")
    """, {"LD_PRELOAD": f"{asan}:{ubsan}", "LSH_ORACLE_LIB": lib})
    assert res.returncode == 0 and "ok" in res.stdout, res.stdout[-3000:] + res.stderr[-3000:]
    assert "runtime error" not in res.stderr and "ERROR: AddressSanitizer" not in res.stderr


def test_abi_validation_under_sanitizers(tmp_path):
    objs = [os.path.join(PKG, "_build", f + ".o")
            for f in ("hash", "sort", "attn_fwd", "attn_bwd", "combine", "dense", "block")]
    if not all(os.path.exists(o) for o in objs):
        pytest.skip("kernel objects not built (run __graft_entry__.build())")
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    rt = glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so")
    if not os.path.exists(hipcc) or not rt:
        pytest.skip("hipcc or the clang sanitizer runtime is missing")
    san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-sanitize-recover=undefined"]
    api_objs = []
    for src in ("lsh_api.cpp", "block_api.cpp"):
        o = str(tmp_path / (src + ".san.o"))
        subprocess.check_call([hipcc, "-O1", "-g", "-std=c++17", "-fPIC", "--offload-arch=gfx950", *san,
                               "-I", os.path.join(ROOT, "include"), "-I", os.path.join(PKG, "csrc"),
                               "-c", os.path.join(PKG, "csrc", src), "-o", o])
        api_objs.append(o)
    lib = str(tmp_path / "liblsh_san.so")
    subprocess.check_call([hipcc, "--offload-arch=gfx950", "-shared", "-fPIC", *san, "-shared-libasan",
                           *api_objs, *objs, "-o", lib])
    res = _run(f"""
        import ctypes, os
        from paper_2001_04451_amd import lsh
        lsh.LIB_PATH = {lib!r}
        L = lsh.lib()
        FAKE = ctypes.c_void_p(0x1000)
        def cfg(**kw):
            base = dict(B=1, H=2, L=1024, d=64, n_buckets=64, n_rounds=2, chunk=64, causal=0,
                        scale=0.125, self_mask=1e5)
            base.update(kw)
            return lsh.LshConfig(**base)
        for bad in (dict(B=0), dict(L=0), dict(n_buckets=7), dict(n_rounds=0), dict(chunk=0),
                    dict(scale=float("nan")), dict(chunks_after=-1)):
            c = cfg(**bad)
            assert L.lsh_hash(ctypes.byref(c), 1, FAKE, FAKE, FAKE, FAKE, 1 << 30, None) == -1
            assert L.lsh_workspace_bytes(ctypes.byref(c), 1, lsh.LSH_OP_FORWARD) == 0
        for unsup in (dict(d=32), dict(n_buckets=2048), dict(n_rounds=17), dict(chunk=96),
                      dict(self_mask=10.0), dict(chunks_after=2), dict(attend_across=1)):
            c = cfg(**unsup)
            n = L.lsh_workspace_bytes(ctypes.byref(c), 1, lsh.LSH_OP_FORWARD)
            assert L.lsh_attention_fwd(ctypes.byref(c), 1, FAKE, FAKE, FAKE, FAKE, None, FAKE,
                                       FAKE, FAKE, FAKE, FAKE, n, None) == -2
        c = cfg()
        for op in range(7):
            L.lsh_workspace_bytes(ctypes.byref(c), 1, op)
        n = L.lsh_workspace_bytes(ctypes.byref(c), 1, lsh.LSH_OP_ATTN_BWD)
        args = [FAKE] * 12
        args[3] = ctypes.c_void_p(0x1008)
        assert L.lsh_chunk_attn_bwd(ctypes.byref(c), 1, *args, n, None) == -1
        big = cfg(B=8, H=16, L=65536, n_buckets=1024, n_rounds=8)
        assert L.lsh_sort_permute_static(ctypes.byref(big), FAKE, FAKE, FAKE, FAKE, None) == -2
        # the reversible block's validation
        bc = lsh.BlockConfigC(cfg(), 256, 64, 1e-5)
        for op in range(3):
            assert L.lsh_block_workspace_bytes(ctypes.byref(bc), op) > 0
        w = lsh.BlockWeightsC(*([FAKE.value] * 12))
        assert L.lsh_rev_attention(ctypes.byref(bc), ctypes.byref(w), FAKE, None, FAKE, 1.0, FAKE, 16,
                                   None) == -1
        assert L.lsh_rev_feed_forward(ctypes.byref(lsh.BlockConfigC(cfg(), 100, 0, 1e-5)), ctypes.byref(w),
                                      FAKE, None, FAKE, 1.0, FAKE, 1 << 40, None) == -2
        assert L.lsh_linear_bf16(128, 100, 64, FAKE, FAKE, None, None, 1.0, FAKE, None, None) == -2
        for s in (0, -1, -2, -3, 5):
            L.lsh_status_string(s)
        print("ok")
    """, {"LD_PRELOAD": rt[0]})
    assert res.returncode == 0 and "ok" in res.stdout, res.stdout[-3000:] + res.stderr[-3000:]
    assert "runtime error" not in res.stderr and "ERROR: AddressSanitizer" not in res.stderr
