"""The C ABI's host validation layer (csrc/abi.hip) built under AddressSanitizer and
UndefinedBehaviorSanitizer and driven by tests/sanitize/abi_harness.cpp, whose stub launchers
record their arguments instead of launching kernels: no GPU is used. The harness calls every
entry point with valid and invalid arguments; the sanitizers must report nothing."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2608_05448_amd", "csrc")
HARNESS = os.path.join(ROOT, "tests", "sanitize", "abi_harness.cpp")
ROCM = "/opt/rocm"


def _tools():
    hipcc = shutil.which("hipcc") or os.path.join(ROCM, "bin", "hipcc")
    clang = os.path.join(ROCM, "llvm", "bin", "clang++")
    if not (os.path.exists(hipcc) and os.path.exists(clang)):
        pytest.skip("ROCm compilers not found")
    return hipcc, clang


def test_abi_validation_layer_is_clean_under_asan_and_ubsan(tmp_path):
    hipcc, clang = _tools()
    # The sanitizer flags apply to the host pass alone (-Xarch_host); device code is unchanged.
    flags = ["-O1", "-g", "-fno-omit-frame-pointer", "-std=c++17", "--offload-arch=gfx950",
             "-Xarch_host", "-fsanitize=address", "-Xarch_host",
             "-fsanitize=undefined", "-Xarch_host", "-fno-sanitize-recover=undefined",
             f"-I{os.path.join(ROOT, 'include')}"]
    objs = []
    for src in (os.path.join(CSRC, "abi.hip"), HARNESS):
        obj = str(tmp_path / (os.path.basename(src) + ".o"))
        cmd = [hipcc, *flags, "-x", "hip", "-c", src, "-o", obj]
        r = subprocess.run(cmd, capture_output=True, text=True)
        assert r.returncode == 0, r.stdout + r.stderr
        objs.append(obj)
    exe = str(tmp_path / "abi_harness")
    r = subprocess.run([clang, "-fsanitize=address,undefined", *objs, f"-L{ROCM}/lib",
                        "-lamdhip64", f"-Wl,-rpath,{ROCM}/lib", "-lpthread", "-o", exe],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stdout + r.stderr
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0:halt_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=120)
    print(r.stdout, r.stderr)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "all checks passed" in r.stdout
    assert "runtime error" not in r.stderr and "AddressSanitizer" not in r.stderr
    # The instrumentation is live: a planted out-of-bounds read in the harness is reported.
    r = subprocess.run([exe, "--plant-overflow"], capture_output=True, text=True, env=env,
                       timeout=120)
    assert r.returncode != 0 and "heap-buffer-overflow" in r.stderr
