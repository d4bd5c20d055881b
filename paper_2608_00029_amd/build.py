"""Build the HIP attention library (libcattn.so) in-tree for gfx950.

Every .hip file under csrc/ is compiled with hipcc for gfx950 only, in
parallel, then linked into paper_2608_00029_amd/libcattn.so.  Packed fp32 ALU
instructions are disabled for all device code.

build_test_library() links a second library for the test suite only,
libcattn_noclamp.so: the same objects except that the bf16 attention kernels
are compiled with CATTN_TEST_NOCLAMP=1 (every tile visited, the ones past the
causal diagonal fully masked), so that a GPU test can show that the causal loop
clamping changes no result.  Nothing in the package loads it.
"""

from __future__ import annotations

import concurrent.futures as cf
import glob
import os
import shutil
import subprocess

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIB = os.path.join(PKG, "libcattn.so")
NOCLAMP_LIB = os.path.join(PKG, "libcattn_noclamp.so")
OBJ_DIR = os.path.join(PKG, "_build")

ARCH = "gfx950"
HIPCC_FLAGS = [
    f"--offload-arch={ARCH}",
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-Wall",
    "-Wno-unused-function",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # keep matrix-core accumulators in ordinary VGPRs: the softmax rescale and
    # the epilogue then read them directly instead of copying through AGPRs
    "-mllvm", "-amdgpu-mfma-vgpr-form",
    "-I", os.path.join(ROOT, "include"),
]


def _hipcc() -> str:
    p = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(p):
        raise RuntimeError("hipcc not found (ROCm is required to build the library)")
    return p


def _run(cmd):
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    # hipcc's host pass warns that it does not know the packed-fp32 feature: harmless.
    lines = [ln for ln in r.stdout.splitlines() if "packed-fp32-ops" not in ln]
    return r.returncode, "\n".join(lines)


def _compile(cmds, jobs, verbose):
    with cf.ThreadPoolExecutor(max_workers=max(1, min(jobs, len(cmds)))) as ex:
        results = list(ex.map(_run, cmds))
    for cmd, (rc, msg) in zip(cmds, results):
        if verbose and msg.strip():
            print(msg)
        if rc != 0:
            raise RuntimeError(f"hipcc failed ({rc}): {' '.join(cmd)}\n{msg}")


def _link(hipcc, out, objs, verbose):
    tmp = out + ".tmp"
    rc, msg = _run([hipcc, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs])
    if rc != 0:
        raise RuntimeError(f"link failed ({rc}):\n{msg}")
    os.replace(tmp, out)
    if verbose:
        print(f"built {out}")


def _sources():
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip")))
    if not srcs:
        raise RuntimeError(f"no HIP sources under {CSRC}")
    return srcs


def _obj(src, tag=""):
    return os.path.join(OBJ_DIR, os.path.basename(src) + tag + ".o")


def build(verbose: bool = False, jobs: int = 8) -> str:
    """Compile every source and link libcattn.so; return its path.  Always rebuilds."""
    hipcc = _hipcc()
    os.makedirs(OBJ_DIR, exist_ok=True)
    srcs = _sources()
    _compile([[hipcc, *HIPCC_FLAGS, "-c", s, "-o", _obj(s)] for s in srcs], jobs, verbose)
    _link(hipcc, LIB, [_obj(s) for s in srcs], verbose)
    return LIB


def build_test_library(verbose: bool = False) -> str:
    """Link libcattn_noclamp.so from build()'s objects and a no-clamp compile of
    the bf16 attention kernels; return its path.  Run build() first."""
    hipcc = _hipcc()
    srcs = _sources()
    bf16 = os.path.join(CSRC, "attn_bf16.hip")
    _compile([[hipcc, *HIPCC_FLAGS, "-DCATTN_TEST_NOCLAMP=1", "-c", bf16, "-o", _obj(bf16, ".noclamp")]], 1, verbose)
    objs = [_obj(s, ".noclamp") if s == bf16 else _obj(s) for s in srcs]
    for o in objs:
        if not os.path.exists(o):
            raise RuntimeError(f"{o} is missing: run build() first")
    _link(hipcc, NOCLAMP_LIB, objs, verbose)
    return NOCLAMP_LIB


if __name__ == "__main__":
    build(verbose=True)
    build_test_library(verbose=True)
