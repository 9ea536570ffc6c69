"""The C ABI from C (CPU): include/bfla.h compiles on its own as C99 and as
C++11 with every warning an error, and a plain C host program
(tests/c_abi/bfla_c_driver.c, HIP runtime C API only) compiles against it and
links with libbfla.so.  tests/test_gpu_c_abi.py runs that program."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
INCLUDE = os.path.join(ROOT, "include")
SRC = os.path.join(ROOT, "tests", "c_abi", "bfla_c_driver.c")
OUT = os.path.join(ROOT, "tests", "c_abi", "_build")
DRIVER = os.path.join(OUT, "bfla_c_driver")
LIBDIR = os.path.join(ROOT, "paper_2605_12193_amd")
ROCM = "/opt/rocm"


def _tool(name):
    path = shutil.which(name)
    if path is None:
        pytest.skip(f"{name} not found")
    return path


def build_driver() -> str:
    """Compile the C driver (gcc, C99, warnings as errors; the HIP headers
    are system headers) and link it with the in-tree libbfla.so."""
    if not os.path.exists(os.path.join(LIBDIR, "libbfla.so")):
        pytest.skip("libbfla.so is not built")
    os.makedirs(OUT, exist_ok=True)
    cmd = [_tool("gcc"), "-std=c99", "-O2", "-Wall", "-Wextra", "-Werror", "-pedantic",
           "-D__HIP_PLATFORM_AMD__", "-isystem", os.path.join(ROCM, "include"), "-I", INCLUDE,
           SRC, "-L", LIBDIR, "-lbfla", "-L", os.path.join(ROCM, "lib"), "-lamdhip64",
           "-Wl,-rpath,$ORIGIN/../../../paper_2605_12193_amd",
           "-Wl,-rpath," + os.path.join(ROCM, "lib"), "-o", DRIVER]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, f"{' '.join(cmd)}\n{r.stderr}"
    return DRIVER


@pytest.mark.parametrize("lang,std,compiler", [("c", "-std=c99", "gcc"),
                                               ("c++", "-std=c++11", "g++")])
def test_header_stands_alone(lang, std, compiler, tmp_path):
    src = tmp_path / ("use." + ("c" if lang == "c" else "cpp"))
    src.write_text('#include "bfla.h"\n'
                   "int probe(void) { bfla_problem p; bfla_params q; bfla_view v; bfla_kv k;\n"
                   "  (void)p; (void)q; (void)v; (void)k;\n"
                   "  return BFLA_OK + BFLA_KV_PAGED + BFLA_WS_EXPAND + (int)BFLA_MAX_BATCH; }\n")
    r = subprocess.run([_tool(compiler), std, "-Wall", "-Wextra", "-Werror", "-pedantic",
                        "-fsyntax-only", "-I", INCLUDE, str(src)], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr


def test_c_driver_compiles_and_links():
    path = build_driver()
    r = subprocess.run([path], capture_output=True, text=True)
    assert r.returncode == 1 and "usage" in r.stderr
