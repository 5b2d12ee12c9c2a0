"""Builds the HIP library libsoap_mi355x.so in-tree with hipcc for gfx950.

Each source is compiled to an object of its own (in parallel, under
``_build/`` at the repository root), then the objects are linked into the
shared library.  ``extra`` flags apply to the compile steps; ``out`` names
another output file (a sanitizer build of the host code, for instance)."""
import glob
import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
LIB = os.path.join(HERE, "libsoap_mi355x.so")
BUILD_DIR = os.path.join(ROOT, "_build")
SOURCES = sorted(glob.glob(os.path.join(HERE, "csrc", "*.hip")))
HEADERS = sorted(glob.glob(os.path.join(HERE, "csrc", "*.h"))) + [
    os.path.join(ROOT, "include", "soap.h")]

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
    # packed-FP32 instructions are kept out of every kernel
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", os.path.join(ROOT, "include"),
]


def stale(out: str = LIB) -> bool:
    if not os.path.exists(out):
        return True
    t = os.path.getmtime(out)
    return any(os.path.getmtime(p) > t for p in SOURCES + HEADERS + [__file__])


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(" ".join(cmd) + "\n" + res.stdout + res.stderr)
    return res.returncode


def build(force: bool = True, verbose: bool = False, extra=(), link_extra=(), out: str = LIB,
          jobs: int = 0) -> str:
    if not force and not stale(out):
        return out
    tag = os.path.splitext(os.path.basename(out))[0]
    objdir = os.path.join(BUILD_DIR, tag)
    os.makedirs(objdir, exist_ok=True)
    os.makedirs(os.path.dirname(os.path.abspath(out)), exist_ok=True)
    objs = [os.path.join(objdir, os.path.basename(src)[:-4] + ".o") for src in SOURCES]
    newest_dep = max(os.path.getmtime(p) for p in HEADERS + [__file__])

    def obj_stale(src, obj):
        return (force or not os.path.exists(obj)
                or os.path.getmtime(obj) < max(newest_dep, os.path.getmtime(src)))

    cmds = [[HIPCC] + FLAGS + list(extra) + ["-c", src, "-o", obj]
            for src, obj in zip(SOURCES, objs) if obj_stale(src, obj)]
    jobs = jobs or max(1, min(len(cmds), 16, os.cpu_count() or 1))
    with ThreadPoolExecutor(max_workers=jobs) as ex:
        codes = list(ex.map(lambda c: _run(c, verbose), cmds))
    if any(codes):
        raise RuntimeError("hipcc failed compiling the sources of %s" % out)
    tmp = out + ".tmp%d" % os.getpid()
    link = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC"] + list(link_extra) + objs + [
        "-o", tmp]
    if _run(link, verbose) != 0:
        raise RuntimeError("hipcc failed linking %s" % out)
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build(force=True, verbose=True, extra=sys.argv[1:]))
