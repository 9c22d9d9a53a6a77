"""Build libavtp.so (HIP kernels for gfx950 + the C-ABI host layer) in-tree.

    python -m paper_2608_26806_amd.build

Every source is compiled by hipcc for gfx950 only; the library lands next to
this file, where the binding loads it.
"""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libavtp.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

SOURCES = ["avtp_api.cpp", "score_attn.hip", "finalize.hip", "score_variation.hip", "budget.hip",
           "select.hip", "compact.hip", "layer_stat.hip", "progressive.hip", "score_noalloc.hip"]

FLAGS = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
         # packed fp32 ALU ops stay off on this target
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-Wall", "-Wno-unused-function", "-Wno-unused-command-line-argument"]


def _compile(src: str, obj: str) -> None:
    cmd = [HIPCC, *FLAGS, "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    noise = "is not a recognized feature for this target"
    err = "\n".join(l for l in (r.stdout + r.stderr).splitlines() if noise not in l)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed on {src}:\n{err}")
    if err.strip():
        print(err, file=sys.stderr)


def build(verbose: bool = True) -> str:
    objdir = os.path.join(HERE, "_build")
    os.makedirs(objdir, exist_ok=True)
    objs = [os.path.join(objdir, os.path.splitext(s)[0] + ".o") for s in SOURCES]
    with ThreadPoolExecutor(max_workers=min(len(SOURCES), os.cpu_count() or 4)) as ex:
        list(ex.map(lambda p: _compile(*p), zip(SOURCES, objs)))
    tmp = LIB + ".tmp"
    cmd = [HIPCC, "-shared", "-fPIC", f"--offload-arch={ARCH}", *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n" + r.stdout + r.stderr)
    os.replace(tmp, LIB)
    if verbose:
        print(f"built {LIB}")
    return LIB


def build_host_sanitized(out_path: str) -> str:
    """A copy of the library whose host validation layer (avtp_api.cpp) is
    built with AddressSanitizer and UndefinedBehaviorSanitizer (host code
    only; the kernels are the regular objects).  Used by the CPU tests, which
    load it with the ASan runtime preloaded.  Builds the regular objects first
    if they are missing."""
    objdir = os.path.join(HERE, "_build")
    objs = [os.path.join(objdir, os.path.splitext(x)[0] + ".o") for x in SOURCES]
    if not all(os.path.exists(o) for o in objs):
        build(verbose=False)
    san_obj = out_path + ".api.o"
    cmd = [HIPCC, "-O1", "-g", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
           "-fno-omit-frame-pointer",
           "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-sanitize-recover=undefined",
           "-c", os.path.join(CSRC, "avtp_api.cpp"), "-o", san_obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("sanitized build of avtp_api.cpp failed:\n" + r.stdout + r.stderr)
    others = [o for o in objs if not o.endswith(os.sep + "avtp_api.o")]
    r = subprocess.run([HIPCC, "-shared", "-fPIC", f"--offload-arch={ARCH}", *others, san_obj,
                        "-o", out_path], capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n" + r.stdout + r.stderr)
    os.remove(san_obj)
    return out_path


if __name__ == "__main__":
    build()
