"""Build libpkv.so (HIP kernels + C ABI) for gfx950 in-tree with hipcc."""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libpkv.so")
SOURCES = ["pkv_kernels.hip", "pkv_capi.cpp", "pkv_host.cpp"]

# Packed-fp32 instructions stay off: plain fp32 ops only (the host pass warns that it
# does not know the feature; that is harmless).
HIP_FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def hipcc() -> str:
    for cand in (shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def build(verbose: bool = False, extra_flags: list[str] | None = None, out: str | None = None) -> str:
    """Compile every source and link libpkv.so next to this file (or at `out`: an A/B
    build with `extra_flags`, loaded through the PKV_LIBRARY environment variable).
    Always recompiles."""
    lib = out or LIB
    tmp = lib + ".tmp"
    cmd = [hipcc(), *HIP_FLAGS, *(extra_flags or []), "-shared", "-o", tmp,
           *[os.path.join(CSRC, s) for s in SOURCES]]
    res = subprocess.run(cmd, cwd=CSRC, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError("hipcc failed:\n" + " ".join(cmd) + "\n" + res.stdout + res.stderr)
    if verbose:
        print(" ".join(cmd))
    os.replace(tmp, lib)
    return lib


if __name__ == "__main__":
    # python build.py [--out PATH] [hipcc flags...]
    argv = sys.argv[1:]
    out = None
    if argv[:1] == ["--out"]:
        out, argv = os.path.abspath(argv[1]), argv[2:]
    print(build(verbose=True, extra_flags=argv, out=out))
