"""Build libim2win.so (HIP kernels + C ABI) for gfx950 with hipcc, in-tree.

Usage: python -m paper_2306_14320_amd.build   (always recompiles)
"""
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libim2win.so")
SOURCES = ["api.hip", "transform.hip", "conv_f32.hip", "conv_bf16.hip", "conv_bf16_image.hip", "conv_f32_band.hip", "conv_plain.hip", "check.hip", "direct.hip"]
ARCH = "gfx950"


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (needs ROCm with gfx950 support)")


def build(verbose: bool = False, jobs: int = 8) -> str:
    """Compile every HIP source for gfx950 and link libim2win.so; returns its path."""
    objdir = os.path.join(PKG, "_build")
    os.makedirs(objdir, exist_ok=True)
    common = [
        "--offload-arch=" + ARCH, "-O3", "-std=c++17", "-fPIC",
        "-I" + INCLUDE, "-I" + CSRC,
        # packed fp32 VALU instructions stay off (their results are not trusted here)
        "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
        "-Wno-unused-command-line-argument",
    ]
    procs = []
    objs = []
    for src in SOURCES:
        obj = os.path.join(objdir, src.replace(".hip", ".o"))
        objs.append(obj)
        cmd = [hipcc()] + common + ["-c", os.path.join(CSRC, src), "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        procs.append(subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True))
        if len(procs) >= jobs:
            _wait(procs.pop(0), verbose)
    for p in procs:
        _wait(p, verbose)
    tmp = LIB + ".tmp"
    link = [hipcc(), "--offload-arch=" + ARCH, "-shared", "-fPIC", "-o", tmp] + objs + [
        "-Wl,-rpath,/opt/rocm/lib", "-Wl,-z,defs"]
    if verbose:
        print(" ".join(link), flush=True)
    subprocess.run(link, check=True)
    os.replace(tmp, LIB)
    return LIB


def _wait(p, verbose):
    out, _ = p.communicate()
    noise = "is not a recognized feature for this target"
    lines = [l for l in out.splitlines() if noise not in l]
    if p.returncode != 0:
        sys.stderr.write("\n".join(lines) + "\n")
        raise RuntimeError(f"hipcc failed ({' '.join(p.args[-3:])})")
    if verbose and lines:
        print("\n".join(lines))


if __name__ == "__main__":
    print(build(verbose=True))
