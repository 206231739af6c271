"""Build libdblast.so (HIP, gfx950) in-tree with hipcc.

    python -m paper_2608_05448_amd.build          # or: from paper_2608_05448_amd import build

Every translation unit is compiled with packed-fp32 instructions disabled; the sampler and
verifier units (every discrete decision of the determinism contract) are also compiled with
floating-point contraction off.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libdblast.so")

ARCH = "gfx950"
SOURCES = {
    "abi.hip": [],
    "head.hip": [],
    "sample.hip": ["-ffp-contract=off"],
    "verify.hip": ["-ffp-contract=off"],
    "greedy.hip": ["-ffp-contract=off"],
    "objective.hip": [],
    "target.hip": ["-ffp-contract=off"],
    "diag.hip": [],
}
COMMON = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}", "-Wall",
          "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
          f"-I{os.path.join(ROOT, 'include')}"]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found: the DBLast library needs ROCm's hipcc to build")


def build(verbose: bool = False, jobs: int = 4, extra_flags=(), out: str = LIB,
          build_dir: str = BUILD) -> str:
    """Compile every HIP source for gfx950 and link the library (libdblast.so by default);
    returns its path. ``extra_flags`` are added to every compile (e.g. tile-size macros)."""
    os.makedirs(build_dir, exist_ok=True)
    cc = hipcc()
    procs, objs = [], []
    for src, extra in SOURCES.items():
        obj = os.path.join(build_dir, src.replace(".hip", ".o"))
        cmd = [cc, *COMMON, *extra, *extra_flags, "-c", os.path.join(CSRC, src), "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        procs.append((src, subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT,
                                            text=True)))
        objs.append(obj)
        while len([p for _, p in procs if p.poll() is None]) >= jobs:
            procs[0][1].wait()
    for src, p in procs:
        log, _ = p.communicate()
        if p.returncode != 0:
            raise RuntimeError(f"hipcc failed on {src}:\n{log}")
        if verbose and log.strip():
            print(log)
    tmp = out + ".tmp"
    cmd = [cc, "-shared", "-fPIC", f"--offload-arch={ARCH}", *objs, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, out)
    return out


TEST_HELPER_SRC = os.path.join(ROOT, "tests", "native", "contract_check.hip")
TEST_HELPER_LIB = os.path.join(ROOT, "tests", "native", "libcontract_check.so")


def build_test_helper(verbose: bool = False) -> str:
    """Compile the GPU test helper (an exhaustive check of the contract's quantised exponential,
    loaded only by the tests) with the library's flags and contraction off."""
    cc = hipcc()
    tmp = TEST_HELPER_LIB + ".tmp"
    cmd = [cc, *COMMON, "-ffp-contract=off", "-shared", TEST_HELPER_SRC, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed on {TEST_HELPER_SRC}:\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, TEST_HELPER_LIB)
    return TEST_HELPER_LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
