"""Build libmsparse.so (gfx950) in-tree with hipcc.

Every HIP translation unit is compiled for gfx950 only, with packed-fp32
instruction selection disabled, and linked into one shared library next to
this file.  Intermediate objects go to _build/.
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
BUILD_DIR = os.path.join(HERE, "_build")
LIB_PATH = os.path.join(HERE, "libmsparse.so")
SOURCES = ["api.hip", "index.hip", "attn_fwd.hip", "attn_bwd.hip", "convert.hip", "estimate.hip", "trace.hip", "peak.hip"]
ARCH = "gfx950"


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def common_flags() -> list[str]:
    return [f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-fvisibility=hidden", "-Wall", "-Wno-unused-function",
            "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def _compile(src: str, build_dir: str = BUILD_DIR, defines=()) -> str:
    obj = os.path.join(build_dir, os.path.splitext(src)[0] + ".o")
    cmd = [hipcc(), *common_flags(), *[f"-D{d}" for d in defines], "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{r.stdout}\n{r.stderr}")
    return obj


def build(jobs: int | None = None, verbose: bool = False, out: str = LIB_PATH, defines=()) -> str:
    """Compile and link libmsparse.so; `defines` are extra -D flags (tuning variants)."""
    build_dir = BUILD_DIR if not defines else os.path.join(BUILD_DIR, "_".join(defines).replace("=", ""))
    os.makedirs(build_dir, exist_ok=True)
    jobs = jobs or min(len(SOURCES), os.cpu_count() or 4, 8)
    with cf.ThreadPoolExecutor(jobs) as ex:
        objs = list(ex.map(lambda src: _compile(src, build_dir, defines), SOURCES))
    tmp = out + ".tmp"
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, out)
    if verbose:
        print(f"built {out}", file=sys.stderr)
    return out


def asan_runtime() -> str:
    """The compiler's AddressSanitizer runtime (to preload into the host process)."""
    import glob
    root = os.path.dirname(os.path.dirname(os.path.realpath(hipcc())))
    cands = sorted(glob.glob(os.path.join(root, "lib", "clang", "*", "lib", "linux", "libclang_rt.asan-x86_64.so")))
    cands += sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    if not cands:
        raise RuntimeError("libclang_rt.asan-x86_64.so not found")
    return cands[0]


def build_asan(out: str | None = None) -> str:
    """A host-AddressSanitizer build of the library: the C ABI's host code
    (argument validation, workspace carving, launch plumbing: api.hip) is
    instrumented for the host only (-Xarch_host), the kernels are the usual
    gfx950 objects.  Load it with the runtime from asan_runtime() preloaded."""
    build_dir = os.path.join(BUILD_DIR, "asan")
    os.makedirs(build_dir, exist_ok=True)
    out = out or os.path.join(build_dir, "libmsparse_asan.so")
    objs = []
    for src in SOURCES:
        obj = os.path.join(build_dir, os.path.splitext(src)[0] + ".o")
        extra = (["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fno-omit-frame-pointer", "-g"]
                 if src == "api.hip" else [])
        cmd = [hipcc(), *common_flags(), *extra, "-c", os.path.join(CSRC, src), "-o", obj]
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError(f"hipcc failed for {src}:\n{r.stdout}\n{r.stderr}")
        objs.append(obj)
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-shared-libasan", "-Xarch_host",
           "-fsanitize=address", *objs, "-o", out]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"asan link failed:\n{r.stdout}\n{r.stderr}")
    return out


if __name__ == "__main__":
    build(verbose=True)
