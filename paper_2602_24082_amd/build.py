"""Builds libppattn.so (HIP kernels for gfx950 + host planner + C ABI) in-tree.

    python -m paper_2602_24082_amd.build          # or build() from Python

Every HIP translation unit is compiled with packed-fp32 instructions disabled
(some of their forms have given wrong results on the target machines) and the
objects are linked into one shared library next to this file.
"""
from __future__ import annotations

import concurrent.futures
import hashlib
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB_NAME = "libppattn.so"
LIB_PATH = os.path.join(PKG, LIB_NAME)
BUILD_DIR = os.path.join(PKG, "_build")
ARCH = "gfx950"

SOURCES = ["pp_host.cpp", "pp_attn_fwd.hip", "pp_attn_bwd.hip", "pp_logprob.hip", "pp_rm.hip", "pp_rope.hip", "pp_stage.hip",
           "pp_noalloc.hip"]

COMMON = [
    "-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wno-unused-command-line-argument",
    f"-I{INCLUDE}", f"-I{CSRC}",
]


def source_digest() -> str:
    """sha256 over the library's sources: every file of csrc/ and the public
    header (names and contents).  Embedded in the library as pp_build_id()."""
    h = hashlib.sha256()
    files = sorted(os.path.join(CSRC, f) for f in os.listdir(CSRC) if not f.startswith("."))
    files.append(os.path.join(INCLUDE, "pp_attn.h"))
    for fn in files:
        if not os.path.isfile(fn):
            continue
        h.update(os.path.basename(fn).encode())
        with open(fn, "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def hipcc() -> str:
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if c and os.path.exists(c):
            return c
    raise RuntimeError("hipcc not found; the HIP library cannot be built")


def _compile(src: str, build_dir: str = BUILD_DIR, defines=()) -> str:
    obj = os.path.join(build_dir, os.path.splitext(src)[0] + ".o")
    cmd = [hipcc(), *COMMON, *[f"-D{d}" for d in defines]]
    if src == "pp_host.cpp":
        cmd.append(f'-DPP_BUILD_ID="{source_digest()}"')
    if src.endswith(".hip"):
        cmd += ["-x", "hip"]
    cmd += ["-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"compiling {src} failed:\n{' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    return obj


def build(verbose: bool = False, defines=(), lib_path: str = LIB_PATH) -> str:
    """Compiles every source and links the shared library; returns its path.

    `defines` (e.g. "PP_FWD_STAGES=3") override the kernels' launch-shape
    defaults in pp_plan.h; with them, pass a `lib_path` outside the package so
    the default library is left alone."""
    build_dir = BUILD_DIR if not defines else lib_path + ".build"
    os.makedirs(build_dir, exist_ok=True)
    with concurrent.futures.ThreadPoolExecutor(max_workers=min(4, len(SOURCES))) as ex:
        objs = list(ex.map(lambda src: _compile(src, build_dir, defines), SOURCES))
    tmp = lib_path + ".tmp"
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"linking failed:\n{' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, lib_path)
    if verbose:
        print(f"built {lib_path}")
    return lib_path


def asan_runtime() -> str:
    """The compiler's shared AddressSanitizer runtime (to preload into a process
    that loads a sanitized library)."""
    r = subprocess.run([hipcc(), "-print-file-name=libclang_rt.asan-x86_64.so"], capture_output=True, text=True)
    path = r.stdout.strip()
    if r.returncode != 0 or not os.path.isabs(path) or not os.path.exists(path):
        raise RuntimeError("AddressSanitizer runtime not found")
    return path


def build_host_sanitized(lib_path: str, verbose: bool = False) -> str:
    """A copy of the library whose host code (validation, planner, staging,
    timing, the C ABI) is built with AddressSanitizer and UndefinedBehaviour-
    Sanitizer; the GPU kernels are the regular ones (no sanitizer runs on GPU
    code here).  Load it with asan_runtime() preloaded, e.g. to run the CPU
    tests of the ABI on it."""
    build_dir = lib_path + ".build"
    os.makedirs(build_dir, exist_ok=True)
    # every sanitizer flag goes to the host compilation only (-Xarch_host before each)
    host_flags = ["-fsanitize=" + kind for kind in ("address", "undefined")]
    host_flags += ["-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer"]
    san = [x for f in host_flags for x in ("-Xarch_host", f)]

    def compile_one(src):
        obj = os.path.join(build_dir, os.path.splitext(src)[0] + ".o")
        cmd = [hipcc(), *COMMON, "-g"]
        if src == "pp_host.cpp":
            cmd += san + [f'-DPP_BUILD_ID="{source_digest()}"']
        else:
            cmd += ["-x", "hip"]
        cmd += ["-c", os.path.join(CSRC, src), "-o", obj]
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError(f"compiling {src} failed:\n{' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
        return obj

    with concurrent.futures.ThreadPoolExecutor(max_workers=min(4, len(SOURCES))) as ex:
        objs = list(ex.map(compile_one, SOURCES))
    tmp = lib_path + ".tmp"
    # the sanitizer runtime is not linked in: the process preloads asan_runtime(),
    # which resolves the instrumentation's symbols when the library is loaded
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"linking failed:\n{' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, lib_path)
    if verbose:
        print(f"built {lib_path}")
    return lib_path


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
