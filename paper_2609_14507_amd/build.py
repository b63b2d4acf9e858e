"""Build the HIP library (libwsk.so) for gfx950 with hipcc, in-tree."""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libwsk.so")
SOURCES = ["wsk_host.cpp", "load.cpp", "policy.cpp", "cpu_attend.cpp", "attend_gqa.hip", "attend_mla.hip", "kernels.hip", "noalloc.hip"]

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    # packed fp32 instructions stay off: hipcc -O3 would otherwise form them
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", os.path.join(ROOT, "include"),
    "-Wno-unused-command-line-argument",
]


# Host-code sanitizers (the device passes are unchanged): AddressSanitizer
# and UndefinedBehaviorSanitizer, for the host-only cache path.  The library
# then needs the clang ASan runtime loaded first (LD_PRELOAD of
# libclang_rt.asan-x86_64.so), since the Python interpreter is not built
# with it.
SANITIZE_FLAGS = [
    "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
    "-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host", "-fno-omit-frame-pointer",
    "-Xarch_host", "-g",
]


def build(verbose: bool = False, sanitize: bool = False) -> str:
    """Compile every source into libwsk.so (always recompiles); sanitize=True
    builds the host code with ASan and UBSan."""
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = [HIPCC] + FLAGS + (SANITIZE_FLAGS if sanitize else []) + [os.path.join(CSRC, s) for s in SOURCES] + \
        ["-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError("hipcc failed building libwsk.so")
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True, sanitize="--sanitize" in sys.argv))
