"""Build libtilefuse.so (HIP for gfx950) in-tree.

    python -m paper_2606_11357_amd.build

Compiles every ``csrc/*.hip`` with hipcc for gfx950 and links one shared
library next to this file.  Always recompiles (it is the "does it build" check).
"""
from __future__ import annotations

import concurrent.futures as cf
import glob
import os
import shutil
import subprocess
import sys
import tempfile

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libtilefuse.so")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-Wall",
    "-Wno-unused-function", "-Wno-unused-command-line-argument",
    # packed fp32 VALU forms stay off on this target
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    f"-I{INCLUDE}", f"-I{CSRC}",
]


# Per-source extra flags.  The 128-row GEMM keeps its MFMA accumulators in
# ordinary VGPRs: with the default AGPR form the register allocator rotates the
# 128 loop-carried accumulators through AGPR copies every K step.  Both GEMMs
# keep small per-thread arrays (group metadata indexed by the unrolled step)
# in registers rather than letting the compiler move them to LDS.
_NO_LDS_PROMOTE = ["-mllvm", "-disable-promote-alloca-to-lds"]
EXTRA = {
    "tf_gemm.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form", *_NO_LDS_PROMOTE],
    # the 256-row GEMM's K step is a fully unrolled 64-slot schedule; let the
    # unroller expand it however large the kernel around it grows
    "tf_gemm256.hip": [*_NO_LDS_PROMOTE, "-mllvm", "-pragma-unroll-threshold=1000000"],
    "tf_gemm_ks.hip": [*_NO_LDS_PROMOTE, "-mllvm", "-pragma-unroll-threshold=1000000"],
}


def _compile(src: str, obj: str, extra=()) -> None:
    cmd = [HIPCC, *FLAGS, *EXTRA.get(os.path.basename(src), []), *extra, "-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {os.path.basename(src)}:\n{r.stderr}")


def _sources():
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip")))
    if not srcs:
        raise RuntimeError("no HIP sources found")
    return srcs


def _build_into(out: str, compile_extra=(), link_extra=()) -> str:
    srcs = _sources()
    tmp = tempfile.mkdtemp(prefix="tf_build_")
    try:
        objs = [os.path.join(tmp, os.path.basename(s) + ".o") for s in srcs]
        with cf.ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
            list(ex.map(lambda so: _compile(so[0], so[1], compile_extra), zip(srcs, objs)))
        out_tmp = out + ".tmp"
        cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *link_extra, "-o", out_tmp, *objs]
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError(f"link failed:\n{r.stderr}")
        os.replace(out_tmp, out)
    finally:
        shutil.rmtree(tmp, ignore_errors=True)
    return out


PROBE_SRC = os.path.join(PKG, "probe", "read_probe.hip")
PROBE_LIB = os.path.join(PKG, "probe", "libtf_read_probe.so")


def build_probe() -> str:
    """The streaming-read probe the benchmark's context figures use (a
    library of its own, not part of libtilefuse)."""
    cmd = [HIPCC, *FLAGS, "-shared", PROBE_SRC, "-o", PROBE_LIB + ".tmp"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for read_probe.hip:\n{r.stderr}")
    os.replace(PROBE_LIB + ".tmp", PROBE_LIB)
    return PROBE_LIB


def build(verbose: bool = False) -> str:
    _build_into(LIB)
    build_probe()
    if verbose:
        print(f"built {LIB} and {PROBE_LIB}")
    return LIB


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
