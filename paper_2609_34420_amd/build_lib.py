"""Build libgtattn.so (HIP, gfx950) in place with hipcc.

    python -m paper_2609_34420_amd.build_lib [-v]

Each .hip source is compiled to an object in parallel, then linked into a
shared library next to this file. Packed-fp32 VALU instructions are disabled
in device code (``-packed-fp32-ops``); the host pass warns that it does not
know that feature, which is harmless.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
from pathlib import Path

PKG = Path(__file__).resolve().parent
CSRC = PKG / "csrc"
LIB = PKG / "libgtattn.so"
BUILD_DIR = PKG / "_build"
SOURCES = ["api.hip", "fwd.hip", "bwd.hip", "bwd_dkdv.hip", "bwd_dq.hip", "bwd_short.hip", "fwd_short.hip", "merge.hip"]
ARCH = os.environ.get("GT_OFFLOAD_ARCH", "gfx950")


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and Path(cand).exists():
            return cand
    raise RuntimeError("hipcc not found (set HIPCC)")


def compile_flags() -> list[str]:
    return [f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
            "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
            "-Wno-unused-result", f"-I{PKG.parent / 'include'}"]


def build(verbose: bool = False, extra: list[str] | None = None) -> Path:
    BUILD_DIR.mkdir(exist_ok=True)
    cc = hipcc()
    flags = compile_flags() + list(extra or [])
    procs = []
    objs = []
    for src in SOURCES:
        obj = BUILD_DIR / (Path(src).stem + ".o")
        cmd = [cc, *flags, "-c", str(CSRC / src), "-o", str(obj)]
        if verbose:
            print(" ".join(cmd), flush=True)
        procs.append((src, subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT)))
        objs.append(obj)
    failed = []
    for src, p in procs:
        out, _ = p.communicate()
        text = out.decode(errors="replace")
        # drop the host pass's notice about the device-only feature flag
        lines = [ln for ln in text.splitlines() if "packed-fp32-ops" not in ln]
        if lines and (verbose or p.returncode != 0):
            print("\n".join(lines), file=sys.stderr)
        if p.returncode != 0:
            failed.append(src)
    if failed:
        raise RuntimeError(f"hipcc failed for {failed}")
    tmp = LIB.with_suffix(".so.tmp")
    cmd = [cc, f"--offload-arch={ARCH}", "-shared", "-fPIC", *map(str, objs), "-o", str(tmp)]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
