"""AddressSanitizer / UndefinedBehaviorSanitizer builds of the CPU code.

Two executables are built in a temporary directory and run:
  * tests/sanitize/oracle_check.c with the oracle's source (both arithmetics:
    double, and the float twin), by gcc with -fsanitize=address,undefined and
    leak checking: every oracle routine over the configuration space;
  * the library's C ABI layer (lq_api.hip, host pass only) by hipcc with the
    sanitizers on the host side, linked with tests/sanitize/api_check.cpp,
    whose stand-in launchers let every validation path run without a GPU.
Any sanitizer report aborts the executable (-fno-sanitize-recover=all), so
the test needs a zero exit status and the driver's own "ok" line.
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = os.path.join(ROOT, "tests", "sanitize")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
CLANG = "/opt/rocm/llvm/bin/clang++"
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0:halt_on_error=1",
           UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1", OMP_NUM_THREADS="2")


def _run(cmd, cwd, **kw):
    r = subprocess.run(cmd, cwd=cwd, capture_output=True, text=True, timeout=300, **kw)
    assert r.returncode == 0, f"{' '.join(cmd)}\n{r.stdout[-4000:]}\n{r.stderr[-4000:]}"
    return r


@pytest.mark.parametrize("real", ["double", "float"])
def test_oracle_under_asan_ubsan(tmp_path, real):
    if shutil.which("gcc") is None:
        pytest.skip("gcc not found")
    exe = str(tmp_path / "oracle_check")
    defs = [] if real == "double" else ["-DOQ_REAL=float", "-DOQ(n)=lqo32_##n"]
    _run(["gcc", "-O1", "-g", "-std=c11", "-fopenmp", "-ffp-contract=off", "-fno-omit-frame-pointer",
          "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-Wall", "-Wextra",
          "-Wno-unused-parameter", *defs, os.path.join(SAN, "oracle_check.c"),
          os.path.join(ROOT, "oracle", "lq_formats.c"), "-o", exe, "-lm"], str(tmp_path))
    r = _run([exe], str(tmp_path), env=ENV)
    assert "oracle sanitizer check ok" in r.stdout


def test_c_abi_host_layer_under_asan_ubsan(tmp_path):
    if not (os.path.exists(HIPCC) and os.path.exists(CLANG)):
        pytest.skip("hipcc / clang++ not found")
    # sanitizers on the host pass only: every -fsanitize option behind -Xarch_host
    flags = ["-x", "hip", "--offload-host-only", "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer",
             "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
             "-Xarch_host", "-fno-sanitize-recover=all",
             "-I", os.path.join(ROOT, "include"), "-I", os.path.join(ROOT, "paper_2609_38166_amd", "csrc")]
    api_o, drv_o, exe = (str(tmp_path / n) for n in ("api.o", "drv.o", "api_check"))
    _run([HIPCC, *flags, "-c", os.path.join(ROOT, "paper_2609_38166_amd", "csrc", "lq_api.hip"), "-o", api_o],
         str(tmp_path))
    _run([HIPCC, *flags, "-c", os.path.join(SAN, "api_check.cpp"), "-o", drv_o], str(tmp_path))
    _run([CLANG, "-fsanitize=address,undefined", api_o, drv_o, "-L/opt/rocm/lib", "-lamdhip64",
          "-Wl,-rpath,/opt/rocm/lib", "-o", exe], str(tmp_path))
    r = _run([exe], str(tmp_path), env=ENV)
    assert "api sanitizer check ok" in r.stdout
