"""Build libscanweaver.so (HIP, gfx950) in place with hipcc.

Usage: ``python -m paper_2606_00601_amd.build`` or ``build()`` from Python.
"""
from __future__ import annotations

import glob
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libscanweaver.so")
ARCH = "gfx950"

# Packed fp32 ops (v_pk_*_f32) are disabled on purpose: the kernels are
# written for scalar fp32 VALU.
HIPCC_FLAGS = [
    "-O3", "-std=c++17", f"--offload-arch={ARCH}", "-fPIC", "-shared", "-fvisibility=hidden",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function",
]


def sources():
    return sorted(glob.glob(os.path.join(CSRC, "*.hip")))


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    # hipcc's host pass does not know the packed-fp32 feature flag; drop that warning
    noise = [ln for ln in res.stderr.splitlines()
             if ln.strip() and "packed-fp32-ops" not in ln and "not a recognized feature" not in ln]
    if res.returncode != 0:
        sys.stderr.write(res.stderr)
        raise RuntimeError("hipcc failed: " + " ".join(cmd[-3:]))
    if noise and verbose:
        sys.stderr.write("\n".join(noise) + "\n")


def build(verbose: bool = False, jobs: int = 0) -> str:
    """Compile every HIP source (one hipcc per translation unit, in parallel;
    each unit's device code is self-contained) and link libscanweaver.so;
    returns its path."""
    import tempfile
    from concurrent.futures import ThreadPoolExecutor
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    compile_flags = [f for f in HIPCC_FLAGS if f != "-shared"]
    jobs = jobs or min(8, os.cpu_count() or 1)
    with tempfile.TemporaryDirectory(prefix="swbuild") as tmpdir:
        objs = []
        cmds = []
        for src in sources():
            obj = os.path.join(tmpdir, os.path.basename(src) + ".o")
            objs.append(obj)
            cmds.append([hipcc, *compile_flags, "-I", INCLUDE, "-I", CSRC, "-c", src, "-o", obj])
        with ThreadPoolExecutor(max_workers=jobs) as ex:
            list(ex.map(lambda c: _run(c, verbose), cmds))
        tmp = LIB + ".tmp%d" % os.getpid()
        _run([hipcc, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs], verbose)
    os.replace(tmp, LIB)
    build_swcall(verbose)
    return LIB


def swcall_path() -> str:
    import sysconfig
    return os.path.join(PKG, "_swcall" + sysconfig.get_config_var("EXT_SUFFIX"))


def build_swcall(verbose: bool = False) -> str:
    """The CPython extension the binding calls the library through
    (csrc/swcall.c, host code only, linked against libscanweaver.so in place)."""
    import sysconfig
    out = swcall_path()
    tmp = out + ".tmp%d" % os.getpid()
    cc = os.environ.get("CC", "gcc")
    cmd = [cc, "-std=c99", "-O2", "-Wall", "-Wextra", "-fPIC", "-shared",
           "-I" + sysconfig.get_paths()["include"], "-I" + INCLUDE,
           os.path.join(CSRC, "swcall.c"), "-L" + PKG, "-lscanweaver", "-Wl,-rpath,$ORIGIN",
           "-o", tmp]
    _run(cmd, verbose)
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build(verbose=True))
