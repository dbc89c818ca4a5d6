"""Compile libpointid.so for gfx950 with hipcc (in-tree, no GPU needed).

    python -m paper_2009_04509_amd.build [-v] [--sanitize address|thread]

Each HIP source under csrc/ is compiled to an object in csrc/_build/, then all
objects are linked into paper_2009_04509_amd/libpointid.so.

--sanitize builds a checking variant of the same library with the host code
instrumented and the device code untouched (every -fsanitize= flag is passed
with -Xarch_host): "address" gives libpointid_asan.so (AddressSanitizer and
UndefinedBehaviorSanitizer, errors fatal), "thread" gives libpointid_tsan.so
(ThreadSanitizer).  Python loads one through the POINTID_LIB environment
variable with the matching runtime preloaded (sanitizer_runtime()).
"""

from __future__ import annotations

import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
OBJDIR = os.path.join(CSRC, "_build")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libpointid.so")

SOURCES = ["api.hip", "batcher.hip", "gather.hip", "conv_fc1_16.hip", "conv_fc1_8.hip", "conv_fc1_f32.hip", "hits.hip",
           "pack.hip", "server.hip", "tail.hip"]

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-Wall",
    # packed fp32 (v_pk_*_f32) code generation stays off for every kernel
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", INCLUDE, "-I", CSRC,
]


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(l for l in r.stdout.splitlines()
                    if "packed-fp32-ops" not in l and "not a recognized feature" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"command failed ({r.returncode}): {' '.join(cmd)}\n{r.stdout}")
    if verbose and out.strip():
        print(out, flush=True)


# host-only sanitizer flags: each -fsanitize= goes to the host compilation
SANITIZE = {
    "address": (["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                 "-Xarch_host", "-fno-sanitize-recover=undefined",
                 "-Xarch_host", "-fno-omit-frame-pointer"],
                ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined"],
                "asan"),
    "thread": (["-Xarch_host", "-fsanitize=thread"], ["-Xarch_host", "-fsanitize=thread"], "tsan"),
}


def library_path(sanitize: str | None = None) -> str:
    return LIB if not sanitize else os.path.join(PKG, f"libpointid_{SANITIZE[sanitize][2]}.so")


def sanitizer_runtime(sanitize: str) -> str | None:
    """The clang runtime a process must preload to load a sanitized build."""
    import glob
    name = {"address": "asan", "thread": "tsan"}[sanitize]
    llvm = os.path.join(os.path.dirname(os.path.dirname(os.path.realpath(HIPCC))), "llvm")
    hits = sorted(glob.glob(os.path.join(llvm, "lib", "clang", "*", "lib", "linux",
                                         f"libclang_rt.{name}-x86_64.so")))
    return hits[-1] if hits else None


def build(verbose: bool = False, jobs: int = 8, sanitize: str | None = None) -> str:
    """Compile every source and link the library; returns the library path."""
    if not os.path.exists(HIPCC):
        raise RuntimeError(f"hipcc not found at {HIPCC}")
    flags, link, objdir = FLAGS, [], OBJDIR
    if sanitize:
        cflags, link, tag = SANITIZE[sanitize]
        # -O1 -g keeps the reports readable; the device code is the same
        flags = [f for f in FLAGS if f != "-O3"] + ["-O1", "-g"] + cflags
        objdir = os.path.join(CSRC, f"_build_{tag}")
    out = library_path(sanitize)
    os.makedirs(objdir, exist_ok=True)
    objs = []
    cmds = []
    for src in SOURCES:
        obj = os.path.join(objdir, os.path.splitext(src)[0] + ".o")
        objs.append(obj)
        cmds.append([HIPCC, *flags, "-c", os.path.join(CSRC, src), "-o", obj])
    with ThreadPoolExecutor(max_workers=max(1, min(jobs, len(cmds)))) as ex:
        list(ex.map(lambda c: _run(c, verbose), cmds))
    tmp = out + ".tmp"
    _run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", *link,
          *(["-shared-libsan"] if sanitize else []), "-o", tmp, *objs], verbose)
    shutil.move(tmp, out)
    return out


if __name__ == "__main__":
    san = sys.argv[sys.argv.index("--sanitize") + 1] if "--sanitize" in sys.argv else None
    path = build(verbose="-v" in sys.argv, sanitize=san)
    print(path)
