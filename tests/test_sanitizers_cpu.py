"""Host AddressSanitizer + UndefinedBehaviorSanitizer runs, CPU only.

* The oracle (oracle/oracle.c) built by gcc with -fsanitize=address,undefined
  and every oracle pin test run against that build.
* libsemshare.so rebuilt with the sanitizers on its host code only (the C ABI
  validation in abi.cpp and the launch code of every kernel file; device code
  is compiled exactly as in the product) and the ABI validation tests run
  against it: every error path that returns before a device call.

Each run is a subprocess with the sanitizer runtime preloaded (Python itself is
not instrumented); an error report fails the test (UBSan is non-recovering)."""
import concurrent.futures
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
GCC_ASAN = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True, text=True).stdout.strip()
CLANG_RT = "/opt/rocm/llvm/lib/clang"


def _clang_asan():
    if not os.path.isdir(CLANG_RT):
        return None
    for ver in sorted(os.listdir(CLANG_RT), reverse=True):
        p = os.path.join(CLANG_RT, ver, "lib", "linux", "libclang_rt.asan-x86_64.so")
        if os.path.exists(p):
            return p
    return None


def _run(code, preload, env_extra=None, timeout=900):
    env = dict(os.environ, LD_PRELOAD=preload, ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1", PYTHONDONTWRITEBYTECODE="1")
    env.update(env_extra or {})
    r = subprocess.run([sys.executable, "-c", code], cwd=ROOT, env=env, capture_output=True, text=True,
                       timeout=timeout)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    assert "runtime error" not in out and "ERROR: AddressSanitizer" not in out, out[-4000:]
    return out


@pytest.mark.skipif(not os.path.isabs(GCC_ASAN) or not os.path.exists(GCC_ASAN), reason="gcc ASan runtime missing")
def test_oracle_under_asan_ubsan(tmp_path):
    lib = str(tmp_path / "liboracle_san.so")
    src = os.path.join(ROOT, "oracle", "oracle.c")
    cmd = ["gcc", "-O1", "-g", "-std=c11", "-fPIC", "-shared", "-fopenmp", "-ffp-contract=off", "-fno-fast-math",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer",
           "-o", lib, src, "-lm"]
    subprocess.run(cmd, check=True)
    code = ("import sys; sys.path.insert(0, 'tests'); import oracle; oracle._LIB_PATH = %r; "
            "import pytest; rc = pytest.main(['-q', '-x', '-p', 'no:cacheprovider', '-m', 'not gpu', "
            "'tests/test_oracle_rope_lsh.py', 'tests/test_oracle_match_gather_select.py', "
            "'tests/test_oracle_prefill.py', 'tests/test_oracle_dynamic.py', 'tests/test_oracle_schedule.py']); "
            "assert oracle._load()._name == %r, 'sanitized oracle not loaded'; sys.exit(rc)") % (lib, lib)
    out = _run(code, GCC_ASAN, {"OMP_NUM_THREADS": "4"})
    assert " passed" in out


@pytest.mark.skipif(_clang_asan() is None, reason="clang ASan runtime missing")
def test_abi_validation_under_asan_ubsan(tmp_path):
    sys.path.insert(0, ROOT)
    from paper_2509_24832_amd import build as B
    san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-sanitize-recover=undefined", "-g"]

    def compile_one(src):
        obj = str(tmp_path / (os.path.basename(src) + ".o"))
        subprocess.run([B.HIPCC, *B.COMMON_FLAGS, *B.EXTRA_FLAGS.get(os.path.basename(src), []), *san,
                        "-x", "hip", "-c", src, "-o", obj], check=True, capture_output=True)
        return obj

    with concurrent.futures.ThreadPoolExecutor(max_workers=8) as ex:
        objs = list(ex.map(compile_one, B.sources()))
    lib = str(tmp_path / "libsemshare_san.so")
    subprocess.run([B.HIPCC, f"--offload-arch={B.ARCH}", "-shared", "-fPIC", "-Xarch_host", "-fsanitize=address",
                    "-Xarch_host", "-fsanitize=undefined", "-shared-libsan", "-o", lib, *objs], check=True,
                   capture_output=True)
    rt = _clang_asan()
    code = ("import sys; sys.path.insert(0, 'tests'); import paper_2509_24832_amd.semshare as b; b.LIB_PATH = %r; "
            "import pytest; rc = pytest.main(['-q', '-x', '-p', 'no:cacheprovider', 'tests/test_abi_cpu.py']); "
            "assert b.load()._name == %r, 'sanitized library not loaded'; sys.exit(rc)") % (lib, lib)
    out = _run(code, rt, {"LD_LIBRARY_PATH": os.path.dirname(rt) + ":" + os.environ.get("LD_LIBRARY_PATH", "")})
    assert " passed" in out
