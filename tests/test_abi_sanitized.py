"""The C ABI layer under AddressSanitizer and UndefinedBehaviorSanitizer, on
the CPU.  The real host sources (api.cpp, shapes.cpp) are compiled host-only
with both sanitizers and linked with stub launchers (tests/abi_host) that
check each launch descriptor and never touch device memory; a driver then
calls every entry point on the error paths and on seeded random problems in
a process with the sanitizer runtime preloaded.  Any out-of-bounds access,
use of freed memory, signed overflow or other undefined behaviour in the host
code aborts the driver and fails this test."""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2605_12193_amd", "csrc")
HOST = os.path.join(ROOT, "tests", "abi_host")
OUT = os.path.join(HOST, "_build")


def _hipcc():
    for cand in ("/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    return None


def _asan_runtime(hipcc):
    clang = os.path.join(os.path.dirname(os.path.realpath(hipcc)), "..", "llvm", "bin", "clang++")
    for cc in (clang, "/opt/rocm/llvm/bin/clang++"):
        if os.path.exists(cc):
            path = subprocess.run([cc, "-print-file-name=libclang_rt.asan-x86_64.so"],
                                  capture_output=True, text=True).stdout.strip()
            if path and os.path.exists(path):
                return path
    return None


# host-only compilation; each sanitizer flag is scoped to the host pass
SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
       "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer"]


@pytest.fixture(scope="module")
def sanitized_lib():
    hipcc = _hipcc()
    if hipcc is None:
        pytest.skip("hipcc not found")
    rt = _asan_runtime(hipcc)
    if rt is None:
        pytest.skip("clang AddressSanitizer runtime not found")
    os.makedirs(OUT, exist_ok=True)
    objs = []
    for src in (os.path.join(CSRC, "api.cpp"), os.path.join(CSRC, "shapes.cpp"),
                os.path.join(HOST, "stub_launchers.cpp")):
        obj = os.path.join(OUT, os.path.basename(src) + ".o")
        cmd = [hipcc, "-x", "hip", "--offload-host-only", "-O1", "-g", "-fPIC", "-std=c++17",
               "-Wall", "-Wno-unused-function", "-I", os.path.join(ROOT, "include"),
               "-I", CSRC] + SAN + ["-c", src, "-o", obj]
        r = subprocess.run(cmd, capture_output=True, text=True)
        assert r.returncode == 0, f"{' '.join(cmd)}\n{r.stdout}\n{r.stderr}"
        objs.append(obj)
    lib = os.path.join(OUT, "libbfla_host_sanitized.so")
    cmd = [hipcc, "-shared", "-fPIC", "-shared-libasan"] + SAN + objs + ["-o", lib]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, f"{' '.join(cmd)}\n{r.stdout}\n{r.stderr}"
    return lib, rt


def test_abi_layer_under_address_and_ub_sanitizers(sanitized_lib):
    lib, rt = sanitized_lib
    env = dict(os.environ)
    env["LD_PRELOAD"] = rt
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=0:halt_on_error=1:exitcode=86"
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1:exitcode=87"
    r = subprocess.run([sys.executable, os.path.join(HOST, "drive_abi.py"), lib, "3000"],
                       env=env, capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, f"exit {r.returncode}\n{r.stdout[-4000:]}\n{r.stderr[-8000:]}"
    assert "abi driver ok" in r.stdout
    print(r.stdout.strip())


def test_the_sanitizers_are_live(sanitized_lib, tmp_path):
    """A planted heap overflow in a helper built the same way is caught: the
    preloaded runtime and the instrumentation really are in effect."""
    hipcc = _hipcc()
    lib, rt = sanitized_lib
    src = tmp_path / "overflow.cpp"
    src.write_text('#include <stdlib.h>\nextern "C" int poke(int i) {\n'
                   '  volatile char* p = (char*)malloc(16); p[i] = 1; int v = p[0]; free((void*)p);\n'
                   '  return v; }\n')
    so = tmp_path / "liboverflow.so"
    r = subprocess.run([hipcc, "-x", "hip", "--offload-host-only", "-shared", "-fPIC",
                        "-shared-libasan", "-O1"] + SAN + [str(src), "-o", str(so)],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    env = dict(os.environ, LD_PRELOAD=rt,
               ASAN_OPTIONS="detect_leaks=0:halt_on_error=1:exitcode=86")
    code = f"import ctypes; L = ctypes.CDLL({str(so)!r}); L.poke(3); L.poke(16)"
    r = subprocess.run([sys.executable, "-c", code], env=env, capture_output=True, text=True,
                       timeout=120)
    assert r.returncode == 86 and "heap-buffer-overflow" in r.stderr, r.stderr[-2000:]
