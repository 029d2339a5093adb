"""Build the HIP library ``libwino_conv.so`` in-tree for gfx950 with hipcc.

Usage: ``python -m paper_1912_02165_amd.build`` (or ``build()`` from Python).
Each source compiles to an object in parallel (the fused kernel once per built
blocking, from wino_fused_inst.hip), then the objects link into the library,
which is written next to this file so it travels with the source tree.
"""

import os
import re
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(HERE, "libwino_conv.so")
OBJDIR = os.path.join(HERE, "_build")
SOURCES = [os.path.join(CSRC, f) for f in (
    "wino_kernels.hip", "fft_kernels.hip", "wino_noalloc.hip", "wino_api.cpp", "wino_tune.cpp")]
INST = os.path.join(CSRC, "wino_fused_inst.hip")
ARCH = "gfx950"
FLAGS = ["-O3", "-std=c++17", "-fPIC", "-Wall", "-Werror=return-type",
         # no packed fp32 instructions in generated code
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def hipcc():
    path = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(path):
        raise RuntimeError("hipcc not found; a ROCm toolchain is required to build the library")
    return path


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError("hipcc failed:\n" + " ".join(cmd) + "\n" + res.stdout + res.stderr)
    return res.stdout + res.stderr


def fused_blockings():
    """(m, R, kit, tb, fs, csp) of every WINO_FUSED_BLOCKINGS entry (wino_internal.h)."""
    text = open(os.path.join(CSRC, "wino_internal.h")).read()
    body = text[text.index("#define WINO_FUSED_BLOCKINGS(X)"):]
    body = body[:body.index("\n\n")]
    return [tuple(int(v) for v in m.split(","))
            for m in re.findall(r"X\(([\d,\s]+)\)", body)]


# Host-side address and undefined-behaviour sanitizers (device code is never
# built with them): for the CPU-only sanitizer run of the host tests, which loads
# the library with the sanitizer runtime preloaded.
HOST_SANITIZE = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                 "-Xarch_host", "-fno-omit-frame-pointer", "-Xarch_host", "-g"]


def build(verbose=False, jobs=None, sanitize=False, out=None):
    """Compile every source into LIB, or into `out` (always recompiles).
    sanitize: instrument the host code with ASan and UBSan (the runtime is not
    linked in; preload it when loading the library)."""
    os.makedirs(OBJDIR, exist_ok=True)
    cc = hipcc()
    lib_path = out or LIB
    extra = HOST_SANITIZE if sanitize else []
    tag = "%d" % os.getpid()
    units = [(src, []) for src in SOURCES]
    for m, R, kit, tb, fs, csp in fused_blockings():
        units.append((INST, [f"-DWS_M={m}", f"-DWS_TB={tb}", f"-DWS_FS={fs}", f"-DWS_CSP={csp}"]))
    objs = [os.path.join(OBJDIR, "%s.%d.%s.o" % (os.path.basename(src), i, tag))
            for i, (src, _) in enumerate(units)]
    cmds = [[cc, f"--offload-arch={ARCH}"] + FLAGS + extra + defs + ["-I", INCLUDE, "-I", CSRC, "-c", src, "-o", o]
            for (src, defs), o in zip(units, objs)]
    jobs = jobs or min(len(cmds), max(1, os.cpu_count() or 1))
    tmp = lib_path + ".tmp" + tag
    try:
        with ThreadPoolExecutor(max_workers=jobs) as ex:
            for out in ex.map(lambda c: _run(c, verbose), cmds):
                if verbose and out.strip():
                    print(out, flush=True)
        _run([cc, f"--offload-arch={ARCH}", "-shared", "-fPIC"] + objs + ["-o", tmp], verbose)
        os.replace(tmp, lib_path)
    finally:
        for f in objs + [tmp]:
            if os.path.exists(f):
                os.remove(f)
    return lib_path


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
