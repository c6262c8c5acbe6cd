"""The C oracle, the seeded input generator and the host side of libgspn's C
ABI built with AddressSanitizer and UndefinedBehaviorSanitizer and driven on
the CPU (no GPU needed):

* oracle_driver.c + oracle/gspn_oracle.c + gspn_inputs/gen.c (gcc): every
  direction mask on small ragged shapes, one-pixel grids, one-line scans;
* abi_driver.c + every library source compiled for the host only (hipcc
  --offload-host-only, sanitizers on the host pass), linked with empty
  offload bundles in place of the device code: argument, alignment, overlap
  and workspace checks of every entry point and the workspace queries (the
  dispatch in counting mode) for one shape of every kernel family.

A sanitizer report or an unexpected status fails the driver's exit status.
"""
import os
import shutil
import subprocess
from concurrent.futures import ThreadPoolExecutor

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HERE = os.path.join(ROOT, "tests", "sanitize")
CSRC = os.path.join(ROOT, "paper_2606_00746_amd", "csrc")
ROCM = "/opt/rocm"
SAN_ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")


def _run(cmd, **kw):
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=600, **kw)
    assert r.returncode == 0, f"{' '.join(cmd)}\n{r.stdout[-4000:]}\n{r.stderr[-4000:]}"
    return r


def test_oracle_and_generator_clean_under_sanitizers(tmp_path):
    if shutil.which("gcc") is None:
        pytest.skip("gcc not found")
    exe = str(tmp_path / "oracle_driver")
    _run(["gcc", "-O1", "-g", "-std=c11", "-fno-omit-frame-pointer",
          "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
          os.path.join(HERE, "oracle_driver.c"), os.path.join(ROOT, "oracle", "gspn_oracle.c"),
          os.path.join(ROOT, "gspn_inputs", "gen.c"), "-lm", "-o", exe])
    r = _run([exe], env=SAN_ENV)
    assert "all cases clean" in r.stdout


def _host_objects(tmp_path):
    from paper_2606_00746_amd import build as lib_build
    hipcc = lib_build.hipcc()
    flags = ["--offload-arch=" + lib_build.ARCH, "--offload-host-only", "-O1", "-g", "-fPIC",
             "-std=c++17", "-Xarch_host", "-fsanitize=address", "-Xarch_host",
             "-fsanitize=undefined", "-Xarch_host", "-fno-sanitize-recover=all",
             "-Xarch_host", "-fno-omit-frame-pointer",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
             "-I", os.path.join(ROOT, "include")]

    def one(src):
        obj = str(tmp_path / (os.path.splitext(src)[0] + ".o"))
        _run([hipcc, *flags, "-x", "hip", "-c", os.path.join(CSRC, src), "-o", obj])
        return obj

    with ThreadPoolExecutor(max_workers=min(8, os.cpu_count() or 1)) as ex:
        return list(ex.map(one, lib_build.SOURCES))


def test_host_abi_clean_under_sanitizers(tmp_path):
    clang = os.path.join(ROCM, "llvm", "bin", "clang")
    if not os.path.exists(clang):
        pytest.skip("ROCm clang not found")
    objs = _host_objects(tmp_path)
    # the host objects name one offload bundle each; with no device code the
    # bundles are empty, and nothing here launches a kernel
    nm_tool = shutil.which("nm") or shutil.which("llvm-nm")
    if nm_tool is None:
        pytest.skip("nm not found")
    nm = _run([nm_tool, "-u", *objs]).stdout
    syms = sorted({ln.split()[-1] for ln in nm.splitlines() if "__hip_fatbin_" in ln})
    stub = tmp_path / "bundles.c"
    stub.write_text("".join(f'const char {s}[32] __attribute__((aligned(4096))) = '
                            f'"__CLANG_OFFLOAD_BUNDLE__";\n' for s in syms))
    san = ["-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
           "-fno-sanitize-recover=all"]
    drv = str(tmp_path / "abi_driver.o")
    _run([clang, *san, "-std=c11", "-Wall", "-Wextra", "-Werror", "-I",
          os.path.join(ROOT, "include"), "-c", os.path.join(HERE, "abi_driver.c"), "-o", drv])
    _run([clang, "-c", str(stub), "-o", str(tmp_path / "bundles.o")])
    exe = str(tmp_path / "abi_driver")
    _run([os.path.join(ROCM, "llvm", "bin", "clang++"), *san, "-o", exe, drv, *objs,
          str(tmp_path / "bundles.o"), "-L" + os.path.join(ROCM, "lib"), "-lamdhip64",
          "-Wl,-rpath," + os.path.join(ROCM, "lib")])
    r = _run([exe], env=SAN_ENV)
    assert "all checks clean" in r.stdout
