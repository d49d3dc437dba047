"""Build step of the HeadCast library: compiles the HIP sources for gfx950 into
an in-tree shared library, paper_2607_20125_amd/libheadcast.so.

    python -m paper_2607_20125_amd.build
"""
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIB = os.path.join(PKG, "libheadcast.so")
SOURCES = ["hc_runtime.cpp", "hc_dense.hip", "hc_spatial.hip", "hc_cache.hip", "hc_static.hip"]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (ROCm is required to build the HeadCast library)")


def build_library(verbose: bool = False) -> str:
    """Compiles every source to an object (in parallel), then links the library."""
    import concurrent.futures
    import tempfile
    flags = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
             # keep the compiler from forming packed fp32 instructions
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
             # MFMA results in vector registers (the online-softmax rescale works on them)
             "-mllvm", "-amdgpu-mfma-vgpr-form",
             # no NaN is produced on these paths: max needs no NaN canonicalisation
             "-fno-honor-nans",
             "-I" + os.path.join(ROOT, "include"), "-I" + CSRC]
    tmp = LIB + ".tmp"

    def run(cmd):
        if verbose:
            print(" ".join(cmd), flush=True)
        res = subprocess.run(cmd, capture_output=True, text=True)
        msgs = [ln for ln in (res.stdout + res.stderr).splitlines() if "packed-fp32-ops" not in ln]
        if res.returncode != 0:
            raise RuntimeError("hipcc failed:\n" + "\n".join(msgs))
        if verbose and msgs:
            print("\n".join(msgs))

    with tempfile.TemporaryDirectory(prefix="headcast_build_") as tdir:
        objs = [os.path.join(tdir, src + ".o") for src in SOURCES]
        cmds = [[hipcc()] + flags + ["-c", os.path.join(CSRC, src), "-o", obj]
                for src, obj in zip(SOURCES, objs)]
        with concurrent.futures.ThreadPoolExecutor(max_workers=len(cmds)) as ex:
            list(ex.map(run, cmds))
        run([hipcc(), "--offload-arch=gfx950", "-shared", "-fPIC"] + objs + ["-o", tmp])
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build_library(verbose="-v" in sys.argv))
