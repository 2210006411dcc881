"""Build libtopkv.so and libtopkv_ceiling.so (HIP, gfx950) in-tree with hipcc.

    python -m paper_2607_28633_amd.build   # -> paper_2607_28633_amd/libtopkv.so, libtopkv_ceiling.so

``build_library(defines=..., out=...)`` builds a variant with extra -D
defines (TOPKV_VPT, TOPKV_WG_PER_CU, TOPKV_NONTEMPORAL) to another path, for
launch-shape sweeps.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
SOURCES = [os.path.join(PKG, "csrc", n) for n in ("topkv.hip", "check.hip", "kvcache1.hip", "dma.hip", "reshard.hip",
                                                        "state.hip")]
CEILING_SOURCES = [os.path.join(PKG, "csrc", "ceiling.hip")]
INCLUDE = os.path.join(ROOT, "include")
LIBRARY = os.path.join(PKG, "libtopkv.so")
CEILING_LIBRARY = os.path.join(PKG, "libtopkv_ceiling.so")
ARCH = "gfx950"


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (ROCm is required to build libtopkv.so)")


def build_command(out: str = LIBRARY, defines=None, sources=None):
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-shared",
           # packed-FP32 instructions are kept out of every kernel
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-Wall", f"-I{INCLUDE}", "-o", out]
    for k, v in (defines or {}).items():
        cmd.append(f"-D{k}={v}")
    if sources is not None:
        return cmd + list(sources)
    return cmd + SOURCES + ["-L/opt/rocm/lib", "-lhsa-runtime64"]


def build_ceiling(out: str = CEILING_LIBRARY, verbose: bool = False) -> str:
    """Compile the measurement kernels' library and return its path."""
    return build_library(out, verbose=verbose, sources=CEILING_SOURCES)


def build_library(out: str = LIBRARY, defines=None, verbose: bool = False, sources=None) -> str:
    """Compile the library (always; no up-to-date check) and return its path."""
    tmp = out + ".tmp"
    cmd = build_command(tmp, defines, sources)
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    noise = ("packed-fp32-ops", "argument unused during compilation")
    msgs = [ln for ln in (res.stdout + res.stderr).splitlines() if ln and not any(x in ln for x in noise)]
    if res.returncode != 0:
        raise RuntimeError("hipcc failed:\n" + "\n".join(msgs))
    if verbose and msgs:
        print("\n".join(msgs))
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build_library(verbose="-v" in sys.argv))
    print(build_ceiling(verbose="-v" in sys.argv))
