"""Host code under AddressSanitizer (no GPU): the CPU oracle, and the C ABI's
host-side validation of libclq.so, rebuilt with ASan and driven in a child
process with the sanitizer runtime preloaded.  Device code is compiled as
usual (the sanitizer applies to the host side only)."""
import os
import subprocess
import sys
import textwrap

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


def _runtime(cmd):
    try:
        p = subprocess.run(cmd, capture_output=True, text=True, check=True).stdout.strip()
    except (OSError, subprocess.CalledProcessError):
        return None
    return p if os.path.isabs(p) and os.path.exists(p) else None


def _child(code, preload, env_extra=None):
    env = dict(os.environ, LD_PRELOAD=preload, ASAN_OPTIONS="detect_leaks=0:abort_on_error=0:exitcode=23")
    env.update(env_extra or {})
    return subprocess.run([sys.executable, "-c", textwrap.dedent(code)], capture_output=True, text=True,
                          env=env, cwd=ROOT, timeout=600)


def test_oracle_under_asan(tmp_path):
    asan = _runtime(["gcc", "-print-file-name=libasan.so"])
    if asan is None:
        pytest.skip("gcc's ASan runtime is not available")
    lib = str(tmp_path / "libclq_oracle_asan.so")
    # the oracle's own flags plus the sanitizer (gcc, host code only)
    subprocess.run(["gcc", "-O1", "-g", "-fopenmp", "-ffp-contract=off", "-std=c11", "-fPIC", "-shared",
                    "-fsanitize=address", "-fno-omit-frame-pointer",
                    os.path.join(ROOT, "oracle", "clq_oracle.c"), "-o", lib, "-lm"], check=True)
    r = _child(f"""
        import numpy as np, oracle, workloads
        oracle._LIB_PATH = {lib!r}
        oracle._lib = None
        for K, b in ((64, 32), (1152, 64), (384, 128)):
            X = workloads.activations(5, K, "L1", seed=K)
            W = workloads.weights(7, K, seed=K + 1)
            perm = workloads.random_perm(K, seed=K + 2)
            r = oracle.linear(X, W, workloads.bias(7, seed=3), b, perm)
            assert np.array_equal(oracle.unpack(r["xq"], K), r["xcodes"])
            oracle.linear(X, W, None, b, wbits=8, abits=8)
        assert {lib!r} in open("/proc/self/maps").read()
        print("asan-oracle-ok")
    """, asan)
    assert r.returncode == 0 and "asan-oracle-ok" in r.stdout, r.stdout[-2000:] + r.stderr[-4000:]


def test_library_host_validation_under_asan(tmp_path):
    asan = _runtime([os.path.join(os.path.dirname(os.path.realpath(HIPCC)), "..", "lib", "llvm", "bin", "clang"),
                     "-print-file-name=libclang_rt.asan-x86_64.so"])
    if asan is None:
        asan = _runtime(["/opt/rocm/lib/llvm/bin/clang", "-print-file-name=libclang_rt.asan-x86_64.so"])
    if asan is None or not os.path.exists(HIPCC):
        pytest.skip("hipcc or clang's ASan runtime is not available")
    sys.path.insert(0, os.path.join(ROOT, "paper_2509_24416_amd"))
    import importlib.util
    spec = importlib.util.spec_from_file_location("_clq_build_asan", os.path.join(ROOT, "paper_2509_24416_amd", "build.py"))
    b = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(b)
    lib = str(tmp_path / "libclq_asan.so")
    # the sanitizer on the host side of every source only
    b.build(extra_flags=["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fno-omit-frame-pointer"],
            out=lib, objdir=str(tmp_path / "objs"))
    r = _child(f"""
        import ctypes
        L = ctypes.CDLL({lib!r})
        i64, i32, f32, p = ctypes.c_int64, ctypes.c_int32, ctypes.c_float, ctypes.c_void_p
        L.clq_status_string.restype = ctypes.c_char_p
        for c in range(-1, 10):
            L.clq_status_string(c)
        A = p(0x10000)
        L.clq_rotate_quant_act.argtypes = [p, i64, p, i64, i64, i32, p, p, p]
        assert L.clq_rotate_quant_act(None, 1152, None, 4, 1152, 64, A, A, None) == 1
        assert L.clq_rotate_quant_act(A, 1152, None, 4, 1152, 48, A, A, None) == 3
        L.clq_w4a4_linear.argtypes = [p, p, p, p, p, i64, i64, i64, p, i64, p, ctypes.c_size_t, p]
        assert L.clq_w4a4_linear(A, A, A, A, None, 8, 8, 96, A, 8, None, 0, None) == 2
        L.clq_w4a4_schedule.argtypes = [i64, i64, i64, i32, p]
        info = (ctypes.c_int64 * 5)()
        for M, N, K in ((1, 1, 64), (43200, 3456, 1152), (16384, 1152, 4608), (2**31 - 1, 8, 64)):
            assert L.clq_w4a4_schedule(M, N, K, 1, ctypes.cast(info, p)) == 0
        L.clq_w4a4_rq_schedule.argtypes = [i64, i64, i64, i32, i32, p]
        info4 = (ctypes.c_int64 * 4)()
        assert L.clq_w4a4_rq_schedule(1024, 1152, 1152, 64, 1, ctypes.cast(info4, p)) == 0
        L.clq_debug_set.argtypes = [i32, i64]
        assert L.clq_debug_set(1, 5) == 0 and L.clq_debug_set(1, 1 << 22) == 0
        L.clq_obs_workspace_bytes.argtypes = [i64, i64, i32]
        L.clq_obs_workspace_bytes.restype = ctypes.c_size_t
        assert L.clq_obs_workspace_bytes(4096, 1152, 3) > 0
        assert {lib!r} in open("/proc/self/maps").read()
        print("asan-lib-ok")
    """, asan)
    assert r.returncode == 0 and "asan-lib-ok" in r.stdout, r.stdout[-2000:] + r.stderr[-4000:]
