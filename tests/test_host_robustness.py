"""Host-side robustness of the C ABI, on the CPU: allocation failures turn
into PEEK_ERR_OUT_OF_MEMORY with no handle produced, and the host code
(libpeek's host side and the oracle) runs clean under AddressSanitizer and
UndefinedBehaviorSanitizer over the CPU tests that exercise it."""
import glob
import os
import shutil
import subprocess
import sys
import textwrap

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = "/opt/rocm/bin/hipcc"


def _asan_runtime():
    hits = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    return hits[-1] if hits else None


def test_allocation_failure_reports_out_of_memory(tmp_path):
    """Host allocations of 8 MiB and more refused while a 2M-node
    description is flattened and while sequences are merged into a tree:
    both calls report OUT_OF_MEMORY, the cache handle stays untouched, the
    library stays usable once allocations succeed again."""
    if shutil.which("gcc") is None:
        pytest.skip("gcc not found")
    shim = tmp_path / "libfailalloc.so"
    subprocess.check_call(["gcc", "-O2", "-shared", "-fPIC", "-o", str(shim), os.path.join(ROOT, "tests", "failalloc.c")])
    script = textwrap.dedent("""
        import ctypes, sys
        import numpy as np
        shim = ctypes.CDLL(sys.argv[1])
        shim.failalloc_arm.argtypes = [ctypes.c_size_t]
        shim.failalloc_refused.restype = ctypes.c_long
        import paper_2607_02525_amd as P
        lib = P._lib
        nn = 2_000_000   # a star: every node but the root a leaf with a one-token edge
        parent = np.zeros(nn, np.int32); parent[0] = -1
        eoff = np.arange(-1, nn, dtype=np.int64); eoff[0] = 0
        etok = np.arange(1, nn, dtype=np.int32)
        canon = np.empty(nn, np.int32)
        i32p, i64p = ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(ctypes.c_int64)
        def build():
            out = ctypes.c_void_p(0x1234)   # must come back untouched
            st = lib.peek_cache_build(nn, parent.ctypes.data_as(i32p), eoff.ctypes.data_as(i64p),
                                      etok.ctypes.data_as(i32p), None, ctypes.byref(out), canon.ctypes.data_as(i32p))
            return st, out.value
        shim.failalloc_arm(8 << 20)
        st, out = build()
        refused = shim.failalloc_refused()
        shim.failalloc_arm(0)
        msg = P.peek_last_error()
        assert st == P.PEEK_ERR_OUT_OF_MEMORY, (st, msg)
        assert out == 0x1234, "no handle on failure"
        assert refused > 0 and "allocation" in msg, (refused, msg)
        # sequences merged into a tree: 300000 distinct sequences of 8 tokens
        seqs = np.arange(300000 * 8, dtype=np.int32)
        offs = np.arange(0, 300001 * 8, 8, dtype=np.int64)
        shim.failalloc_arm(8 << 20)
        try:
            P.peek_tree_from_sequences(seqs, offs)
            raise AssertionError("expected OUT_OF_MEMORY")
        except P.PeekError as e:
            assert e.status == P.PEEK_ERR_OUT_OF_MEMORY, e
        finally:
            shim.failalloc_arm(0)
        # usable again: the same calls now fail only for want of a GPU, or succeed on one
        st, out = build()
        assert st in (P.PEEK_OK, P.PEEK_ERR_UNSUPPORTED_DEVICE, P.PEEK_ERR_DEVICE), (st, P.peek_last_error())
        if st == P.PEEK_OK:
            lib.peek_cache_free(ctypes.c_void_p(out))
        n_nodes = P.peek_tree_from_sequences(seqs, offs)[0].shape[0]
        assert n_nodes == 300001
        print("ok")
    """)
    env = dict(os.environ, LD_PRELOAD=str(shim), PYTHONPATH=ROOT)
    r = subprocess.run([sys.executable, "-c", script, str(shim)], env=env, capture_output=True, text=True,
                       timeout=600, cwd=ROOT)
    assert r.returncode == 0 and r.stdout.strip().endswith("ok"), r.stdout + r.stderr


def test_host_code_under_address_and_undefined_sanitizers(tmp_path):
    """libpeek with its host code built with -fsanitize=address,undefined
    (the device code as usual; no kernel runs on the CPU) and the oracle
    (the same sanitizers) under the C-ABI tests, the oracle tests and the
    eviction-placement tests; any sanitizer report fails the run."""
    rt = _asan_runtime()
    clangxx = "/opt/rocm/llvm/bin/clang++"
    if rt is None or not os.path.exists(HIPCC) or not os.path.exists(clangxx):
        pytest.skip("clang sanitizer runtime or hipcc not found")
    pkg = tmp_path / "paper_2607_02525_amd"
    pkg.mkdir()
    for f in glob.glob(os.path.join(ROOT, "paper_2607_02525_amd", "*.py")):
        shutil.copy(f, pkg)
    san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-omit-frame-pointer"]
    objs = []
    for src in sorted(glob.glob(os.path.join(ROOT, "paper_2607_02525_amd", "csrc", "peek_*.hip"))):
        if os.path.basename(src) == "peek_calib.hip":
            continue
        obj = tmp_path / (os.path.basename(src) + ".o")
        subprocess.check_call([HIPCC, "--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-fPIC",
                               "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
                               "-I" + os.path.join(ROOT, "include"), *san, "-c", src, "-o", str(obj)])
        objs.append(str(obj))
    subprocess.check_call([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", *san, "-o", str(pkg / "libpeek.so"),
                           *objs])
    oracle = tmp_path / "liboracle_san.so"
    subprocess.check_call([clangxx, "-O1", "-g", "-std=c++17", "-shared", "-fPIC", "-fsanitize=address,undefined",
                           "-fno-omit-frame-pointer", "-o", str(oracle), os.path.join(ROOT, "oracle", "oracle.cpp")])
    env = dict(os.environ, LD_PRELOAD=rt, PYTHONPATH=f"{tmp_path}:{ROOT}", PEEK_ORACLE_LIB=str(oracle),
               ASAN_OPTIONS="detect_leaks=0:halt_on_error=1", UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    # run from the scratch directory with pytest appending (not prepending) the
    # repository to sys.path, so the sanitized package is the one imported
    probe = subprocess.run([sys.executable, "-c", "import paper_2607_02525_amd as P; print(P.LIB_PATH)"], env=env,
                           capture_output=True, text=True, timeout=300, cwd=str(tmp_path))
    assert probe.stdout.strip() == str(pkg / "libpeek.so"), probe.stdout + probe.stderr
    check = ("import paper_2607_02525_amd as P, oracle as O; "
             f"assert P.LIB_PATH == {str(pkg / 'libpeek.so')!r}, P.LIB_PATH; "
             f"assert O._LIB == {str(oracle)!r}, O._LIB")
    tests = [os.path.join(ROOT, "tests", f) for f in ("test_abi_cpu.py", "test_oracle.py", "test_evict_placement.py")]
    r = subprocess.run([sys.executable, "-c", check + "; import pytest, sys; sys.exit(pytest.main(sys.argv[1:]))",
                        "-x", "-q", "-s", "-p", "no:cacheprovider", "--import-mode=append", "--rootdir", ROOT,
                        "-m", "not gpu", "-k", "not scale_invariants and not hashed_block_hit", *tests],
                       env=env, capture_output=True, text=True, timeout=1200, cwd=str(tmp_path))
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    assert "ERROR: AddressSanitizer" not in out and "runtime error:" not in out, out[-4000:]
