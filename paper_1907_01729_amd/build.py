"""Build the gfx950 HIP library ``libsinkhorn_hip.so`` in-tree with hipcc.

Each translation unit is compiled to an object in parallel (``_build/``), then
the objects are linked into the shared library.  Every call compiles.
"""
from __future__ import annotations

import glob
import os
import shlex
import shutil
import subprocess
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libsinkhorn_hip.so")
OBJ_DIR = os.path.join(os.path.dirname(HERE), "_build")

# Packed fp32 VALU forms are switched off for all device code (they are not
# needed: the kernels are bound by v_exp_f32 and scalar fp32 VALU issue).
HIP_FLAGS = [
    "-O3", "-std=c++17", "--offload-arch=gfx950", "-fPIC", "-fvisibility=hidden",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wno-unused-command-line-argument",
]


def hipcc() -> str:
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if c and os.path.exists(c):
            return c
    raise RuntimeError("hipcc not found")


def sources():
    return sorted(glob.glob(os.path.join(CSRC, "*.hip")))


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed ({r.returncode}): {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    if verbose and r.stderr.strip():
        print(r.stderr, flush=True)


def _compile_and_link(flags, obj_dir, lib, link_extra=(), verbose=False, jobs=None) -> str:
    os.makedirs(obj_dir, exist_ok=True)
    cc = hipcc()
    srcs = sources()
    objs = [os.path.join(obj_dir, os.path.basename(s)[:-4] + ".o") for s in srcs]
    jobs = jobs or min(len(srcs), max(1, min(16, os.cpu_count() or 1)))
    with ThreadPoolExecutor(max_workers=jobs) as ex:
        futs = [ex.submit(_run, [cc, *flags, "-c", "-o", o, s], verbose) for s, o in zip(srcs, objs)]
        for f in futs:
            f.result()
    tmp = lib + ".tmp"
    _run([cc, *flags, "-shared", *link_extra, "-o", tmp, *objs], verbose)
    os.replace(tmp, lib)
    return lib


def build(verbose: bool = False, jobs: int | None = None) -> str:
    return _compile_and_link(HIP_FLAGS, OBJ_DIR, LIB, verbose=verbose, jobs=jobs)


# Host-side sanitizers for the CPU checks of the C ABI: AddressSanitizer and
# UndefinedBehaviorSanitizer on the host pass only (device code as above),
# the sanitizer runtime linked as a shared library.
HOST_SANITIZE = shlex.split(
    "-Xarch_host -fsanitize=address -Xarch_host -fsanitize=undefined "
    "-Xarch_host -fno-sanitize-recover=all -Xarch_host -fno-omit-frame-pointer")


def build_host_sanitized(verbose: bool = False, jobs: int | None = None) -> str:
    """A copy of the library with sanitized host code, in _build/asan (for
    tests that call only host-side paths of the ABI; never loaded by the
    package)."""
    out = os.path.join(OBJ_DIR, "asan")
    flags = [f if f != "-O3" else "-O1" for f in HIP_FLAGS] + ["-g"] + HOST_SANITIZE
    return _compile_and_link(flags, out, os.path.join(out, "libsinkhorn_hip_asan.so"), link_extra=["-shared-libsan"],
                             verbose=verbose, jobs=jobs)


if __name__ == "__main__":
    print(build(verbose=True))
