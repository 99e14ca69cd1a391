"""Host-side robustness, on the CPU: the oracle built with AddressSanitizer +
UndefinedBehaviorSanitizer and with ThreadSanitizer, and the library's host code
(argument checks, workspace layout, fault injection) built with AddressSanitizer +
UndefinedBehaviorSanitizer on its host pass only, each driven by a small C program
(tests/sanitize/) in a subprocess; and the MPM_FAULT_INJECT=launch hook through the
Python binding. No GPU is touched."""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = os.path.join(ROOT, "tests", "sanitize")
ORACLE_C = os.path.join(ROOT, "oracle", "mpm_oracle.c")
CSRC = os.path.join(ROOT, "paper_2604_05718_amd", "csrc")
HIPCC = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
CLANG = "/opt/rocm/llvm/bin/clang"


def _run(cmd, env=None, cwd=None):
    p = subprocess.run(cmd, capture_output=True, text=True, env=env, cwd=cwd)
    assert p.returncode == 0, f"{' '.join(cmd)}\n{p.stdout[-3000:]}\n{p.stderr[-3000:]}"
    return p.stdout


@pytest.mark.parametrize("san", ["address,undefined", "thread"])
def test_oracle_under_sanitizers(tmp_path, san):
    exe = str(tmp_path / "oracle_driver")
    extra = ["-fno-sanitize-recover=all"] if san != "thread" else []
    _run(["gcc", "-O1", "-g", "-std=c11", f"-fsanitize={san}", *extra, "-fno-omit-frame-pointer",
          "-ffp-contract=off", ORACLE_C, os.path.join(SAN, "oracle_driver.c"), "-lm", "-lpthread", "-o", exe])
    out = _run([exe], env=dict(os.environ, ASAN_OPTIONS="detect_leaks=1", TSAN_OPTIONS="halt_on_error=1"))
    assert "cases ok" in out


@pytest.mark.skipif(not (os.path.exists(HIPCC) and os.path.exists(CLANG)), reason="needs hipcc and ROCm clang")
def test_abi_host_code_under_sanitizers(tmp_path):
    san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-sanitize-recover=all"]
    flags = ["--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-fPIC", "-Xclang", "-target-feature", "-Xclang",
             "-packed-fp32-ops", "-Wno-inline-asm", "-I", os.path.join(ROOT, "include"), "-I", CSRC, *san]
    objs, procs = [], []
    for f in sorted(os.listdir(CSRC)):
        if f.endswith(".hip"):
            o = str(tmp_path / (f[:-4] + ".o"))
            objs.append(o)
            procs.append(subprocess.Popen([HIPCC, *flags, "-c", os.path.join(CSRC, f), "-o", o],
                                          stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True))
    for p in procs:
        out, _ = p.communicate()
        assert p.returncode == 0, out[-3000:]
    drv = str(tmp_path / "abi_driver.o")
    _run([CLANG, "-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-c",
          os.path.join(SAN, "abi_driver.c"), "-o", drv])
    exe = str(tmp_path / "abi_driver")
    _run([HIPCC, "--offload-arch=gfx950", "-fsanitize=address,undefined", drv, *objs, "-o", exe])
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0")  # the HIP runtime's own allocations
    env.pop("MPM_FAULT_INJECT", None)
    assert "abi driver: ok" in _run([exe], env=env)
    env["MPM_FAULT_INJECT"] = "launch"
    assert "injected launch failures" in _run([exe], env=env)


def test_fault_injection_through_the_binding():
    """With MPM_FAULT_INJECT=launch a call that passes its argument checks returns
    MPM_ERR_HIP with hipErrorLaunchFailure, which the binding raises as MPMError."""
    code = r"""
import ctypes
from paper_2604_05718_amd import _lib
lib = _lib.load()
A = ctypes.c_void_p(0x100000)
st = lib.mpm_merge(A, None, None, 2, 16, 64, _lib.MPM_BF16, 0, A, A, None, A, A, 1 << 30, None)
assert st == _lib.MPM_ERR_HIP, st
try:
    _lib.check("mpm_merge", st)
except _lib.MPMError as e:
    assert e.status == _lib.MPM_ERR_HIP and e.hip_error == 719, (e.status, e.hip_error)
    print("raised:", e)
else:
    raise AssertionError("no MPMError")
"""
    env = dict(os.environ, MPM_FAULT_INJECT="launch", PYTHONPATH=ROOT)
    out = _run([sys.executable, "-c", code], env=env, cwd=ROOT)
    assert "MPM_ERR_HIP (hipError_t 719)" in out
