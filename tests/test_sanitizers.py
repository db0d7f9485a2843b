"""Host sanitizer builds (CPU only): the oracle under gcc's AddressSanitizer and
UndefinedBehaviorSanitizer, running every oracle pin, and the library with its
host code under clang's (device code is built as usual and never runs here),
running the C-ABI host-validation tests.  Each run is a child process with the
sanitizer runtime preloaded; UB reports are fatal (-fno-sanitize-recover).  A
control per toolchain shows the runtime is live: a deliberate out-of-bounds
write in a throwaway library must abort with an AddressSanitizer report.
"""
import glob
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer", "-g", "-O1"]
HIPCC = "/opt/rocm/bin/hipcc"
CLANG = "/opt/rocm/llvm/bin/clang"

BAD_C = r"""
#include <stdlib.h>
int bad_write(int n) { int *p = malloc(4 * (size_t)n); p[n] = 1; int r = p[0]; free(p); return r; }
"""


def gcc_asan_runtime():
    p = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True, text=True).stdout.strip()
    return p if os.path.isabs(p) and os.path.exists(p) else None


def clang_asan_runtime():
    c = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    return c[-1] if c else None


def run_child(code, env_extra, timeout=900):
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=1", **env_extra)
    return subprocess.run([sys.executable, "-c", code], cwd=ROOT, env=env, capture_output=True, text=True,
                          timeout=timeout)


def control(compiler, runtime, tmp_path):
    src = tmp_path / "bad.c"
    src.write_text(BAD_C)
    so = tmp_path / "libbad.so"
    subprocess.check_call([compiler, "-shared", "-fPIC", *SAN, "-o", str(so), str(src)])
    r = run_child(f"import ctypes; ctypes.CDLL({str(so)!r}).bad_write(8)", {"LD_PRELOAD": runtime}, timeout=120)
    assert r.returncode != 0 and "AddressSanitizer" in r.stderr, r.stderr[-2000:]


def test_oracle_under_asan_ubsan(tmp_path):
    rt = gcc_asan_runtime()
    if rt is None:
        pytest.skip("gcc has no AddressSanitizer runtime")
    control("gcc", rt, tmp_path)
    so = tmp_path / "libecokv_oracle_san.so"
    subprocess.check_call(["gcc", "-std=c99", "-fPIC", "-shared", "-fopenmp", *SAN, "-o", str(so),
                           os.path.join(ROOT, "oracle", "ecokv_oracle.c"), "-lm"])
    pins = os.path.join(ROOT, "tests", "test_oracle_pins.py")
    code = (f"import sys; sys.path.insert(0, {ROOT!r}); import oracle; oracle.use_library({str(so)!r}); "
            f"import pytest; sys.exit(pytest.main(['-x', '-q', '-p', 'no:cacheprovider', {pins!r}]))")
    r = run_child(code, {"LD_PRELOAD": rt})
    assert r.returncode == 0, (r.stdout[-3000:], r.stderr[-3000:])
    assert "runtime error" not in r.stderr and "AddressSanitizer" not in r.stderr


def test_library_host_code_under_asan_ubsan(tmp_path):
    rt = clang_asan_runtime()
    if rt is None or not os.path.exists(HIPCC):
        pytest.skip("no clang AddressSanitizer runtime or hipcc")
    control(CLANG, rt, tmp_path)
    import importlib.util
    from concurrent.futures import ThreadPoolExecutor
    # the package's build script, for its source list and flags
    spec = importlib.util.spec_from_file_location("ecokv_build", os.path.join(ROOT, "paper_2609_06663_amd", "build.py"))
    B = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(B)
    csrc = os.path.join(ROOT, "paper_2609_06663_amd", "csrc")
    host_san = []
    for f in SAN:  # each host-only flag right after -Xarch_host; device code as usual
        host_san += ["-Xarch_host", f]
    flags = [f for f in B.HIPCC_FLAGS if f != "-O3"]

    def compile_one(src):
        obj = tmp_path / src.replace(".hip", ".o")
        subprocess.check_call([HIPCC, *flags, *host_san, "-c", os.path.join(csrc, src), "-o", str(obj)],
                              stderr=subprocess.DEVNULL)
        return str(obj)

    with ThreadPoolExecutor(max_workers=len(B.SOURCES)) as ex:
        objs = list(ex.map(compile_one, B.SOURCES))
    so = tmp_path / "libecokv_san.so"
    subprocess.check_call([HIPCC, f"--offload-arch={B.ARCH}", "-shared", "-fPIC", *objs, "-o", str(so)])
    abi = os.path.join(ROOT, "tests", "test_abi.py")
    code = (f"import sys; sys.path.insert(0, {ROOT!r}); import paper_2609_06663_amd.ecokv as E; "
            f"assert E._LIB_PATH == {str(so)!r}, E._LIB_PATH; "
            f"import pytest; sys.exit(pytest.main(['-x', '-q', '-p', 'no:cacheprovider', {abi!r}]))")
    r = run_child(code, {"LD_PRELOAD": rt, "ECOKV_LIBRARY": str(so)})
    assert r.returncode == 0, (r.stdout[-3000:], r.stderr[-3000:])
    assert "passed" in r.stdout and "runtime error" not in r.stderr and "AddressSanitizer" not in r.stderr
