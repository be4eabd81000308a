"""A build of libtilefuse with AddressSanitizer and UndefinedBehaviorSanitizer
on its host code (argument checks, layout sizing, planners, launchers), for
CPU tests of the C ABI.  Every sanitizer flag goes to the host compilation
only, so the device code is that of the normal build.

    python -m paper_2606_11357_amd.sanitized_build

The library goes under _build/sanitized/<hash of sources and flags>/ and is
rebuilt only when those change.  A process that loads it must preload the
sanitizer runtime (``runtime()``).
"""
from __future__ import annotations

import glob
import hashlib
import os
import subprocess

from . import build

_OPTS = ("-fsanitize=address", "-fsanitize=undefined", "-fno-sanitize-recover=all",
         "-fno-omit-frame-pointer", "-g", "-O1")
COMPILE = [f for opt in _OPTS for f in ("-Xarch_host", opt)]
LINK = [f for opt in ("-fsanitize=address", "-fsanitize=undefined", "-shared-libsan")
        for f in ("-Xarch_host", opt)]
OUT_DIR = os.path.join(build.ROOT, "_build", "sanitized")


def runtime() -> str:
    """Path of the AddressSanitizer runtime of the toolchain."""
    r = subprocess.run(["/opt/rocm/llvm/bin/clang", "-print-file-name=libclang_rt.asan-x86_64.so"],
                       capture_output=True, text=True, check=True)
    return r.stdout.strip()


def build_sanitized(verbose: bool = False) -> str:
    h = hashlib.sha256()
    files = sorted(glob.glob(os.path.join(build.CSRC, "*.hip")) + glob.glob(os.path.join(build.CSRC, "*.h")))
    for f in files + [os.path.join(build.INCLUDE, "tilefuse.h")]:
        h.update(open(f, "rb").read())
    h.update(" ".join(build.FLAGS + COMPILE + LINK).encode())
    out_dir = os.path.join(OUT_DIR, h.hexdigest()[:16])
    out = os.path.join(out_dir, "libtilefuse_sanitized.so")
    if not os.path.exists(out):
        os.makedirs(out_dir, exist_ok=True)
        build._build_into(out, COMPILE, LINK)
    if verbose:
        print(f"built {out}")
    return out


if __name__ == "__main__":
    build_sanitized(verbose=True)
