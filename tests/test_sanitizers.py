"""The project's host code under AddressSanitizer and UndefinedBehaviorSanitizer
(CPU only): the oracle's C routines, the mesh planner and every argument check
of the C ABI that returns before device work, driven by tests/sanitize/driver.cpp.

Everything sanitized is built with the ROCm clang (one sanitizer runtime):
oracle.c and planner.cpp as host code, abi.hip with the sanitizers on its host
side only (-Xarch_host before each -fsanitize=; its device code and the other
kernels' objects are built as usual).  The driver aborts on the first report."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LLVM = "/opt/rocm/llvm/bin"
HIPCC = "/opt/rocm/bin/hipcc"
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer",
       "-g", "-O1"]
KERNELS = ["gemm.hip", "reduce.hip", "transpose.hip", "attention.hip"]


def _run(cmd, cwd):
    r = subprocess.run(cmd, cwd=cwd, capture_output=True, text=True)
    assert r.returncode == 0, " ".join(cmd) + "\n" + r.stdout[-3000:] + r.stderr[-3000:]
    return r


@pytest.mark.skipif(not (os.path.exists(HIPCC) and os.path.exists(f"{LLVM}/clang++")),
                    reason="ROCm compilers not installed")
def test_host_code_under_asan_and_ubsan(tmp_path):
    inc = ["-I", os.path.join(ROOT, "include")]
    csrc = os.path.join(ROOT, "paper_2301_08658_amd", "csrc")
    objs = []
    o = str(tmp_path / "oracle.o")
    _run([f"{LLVM}/clang", *SAN, "-std=c11", "-ffp-contract=off", "-c",
          os.path.join(ROOT, "oracle", "oracle.c"), "-o", o], tmp_path)
    objs.append(o)
    for src, path in (("planner.cpp", csrc), ("driver.cpp", os.path.join(ROOT, "tests",
                                                                           "sanitize"))):
        o = str(tmp_path / (src + ".o"))
        _run([f"{LLVM}/clang++", *SAN, "-std=c++17", *inc, "-c", os.path.join(path, src), "-o",
              o], tmp_path)
        objs.append(o)
    dev = ["-std=c++17", "-fPIC", "--offload-arch=gfx950", "-Xclang", "-target-feature",
           "-Xclang", "-packed-fp32-ops", *inc]
    host_san = []
    for f in SAN:
        host_san += ["-Xarch_host", f]
    o = str(tmp_path / "abi.o")
    _run([HIPCC, *dev, *host_san, "-c", os.path.join(csrc, "abi.hip"), "-o", o], tmp_path)
    objs.append(o)
    for src in KERNELS:   # reuse the library build's objects when they are there
        built = os.path.join(ROOT, "_build", src.replace(".hip", ".o"))
        o = str(tmp_path / (src + ".o"))
        if os.path.exists(built):
            shutil.copy(built, o)
        else:
            _run([HIPCC, "-O3", *dev, "-c", os.path.join(csrc, src), "-o", o], tmp_path)
        objs.append(o)
    exe = str(tmp_path / "driver")
    _run([f"{LLVM}/clang++", "-fsanitize=address,undefined", "-o", exe, *objs,
          "-L/opt/rocm/lib", "-lamdhip64", "-Wl,-rpath,/opt/rocm/lib", "-lm"], tmp_path)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1", OMP_NUM_THREADS="1")
    r = subprocess.run([exe], cwd=tmp_path, capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode == 0, r.stdout[-3000:] + r.stderr[-5000:]
    assert "sanitized host checks passed" in r.stdout
