"""Build liboctree_nca.so (HIP, gfx950) in-tree with hipcc.

    python -m paper_2508_06993_amd.build

Each .hip file under csrc/ is compiled to an object in parallel, then linked
into paper_2508_06993_amd/liboctree_nca.so.  The library is replaced
atomically, so a process that already loaded the old one keeps working.
Beside it, liboctree_nca.stamp records a hash of the sources, headers and
flags it was built from; ``is_current()`` compares it with the tree.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
import tempfile
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB_NAME = "liboctree_nca.so"
LIB_PATH = os.path.join(PKG, LIB_NAME)
STAMP_PATH = os.path.join(PKG, "liboctree_nca.stamp")
ARCH = "gfx950"

# Packed fp32 VALU instructions are disabled for every device pass: only the
# scalar fp32 forms are emitted.
DEVICE_FLAGS = ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
COMMON_FLAGS = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}", "-I", INCLUDE,
                "-I", CSRC, "-Wall", "-Wno-unused-result"]


def hipcc() -> str:
    path = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(path):
        raise RuntimeError("hipcc not found; a ROCm toolchain is needed to build the library")
    return path


def sources():
    return sorted(os.path.join(CSRC, f) for f in os.listdir(CSRC) if f.endswith(".hip"))


def source_stamp() -> str:
    """sha256 over the library's sources, headers and build flags."""
    import hashlib
    h = hashlib.sha256()
    files = sorted(os.path.join(CSRC, f) for f in os.listdir(CSRC) if f.endswith((".hip", ".h")))
    files += sorted(os.path.join(INCLUDE, f) for f in os.listdir(INCLUDE) if f.endswith(".h"))
    for path in files:
        h.update(os.path.relpath(path, ROOT).encode())
        with open(path, "rb") as f:
            h.update(f.read())
    h.update(" ".join(COMMON_FLAGS + DEVICE_FLAGS).encode())
    return h.hexdigest()


def is_current() -> bool:
    """Whether the built library exists and was built from the sources as they are now."""
    if not os.path.exists(LIB_PATH) or not os.path.exists(STAMP_PATH):
        return False
    with open(STAMP_PATH) as f:
        return f.read().strip() == source_stamp()


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(line for line in res.stdout.splitlines()
                    if "packed-fp32-ops" not in line)   # the host pass does not know the feature
    if res.returncode != 0:
        raise RuntimeError(f"command failed ({res.returncode}): {' '.join(cmd)}\n{out}")
    if verbose and out.strip():
        print(out, flush=True)


def build(verbose: bool = False, jobs: int | None = None) -> str:
    cc = hipcc()
    srcs = sources()
    stamp = source_stamp()
    tmp = tempfile.mkdtemp(prefix="octnca_build_", dir=PKG)
    try:
        objs = [os.path.join(tmp, os.path.basename(s) + ".o") for s in srcs]
        cmds = [[cc, *COMMON_FLAGS, *DEVICE_FLAGS, "-c", s, "-o", o] for s, o in zip(srcs, objs)]
        with ThreadPoolExecutor(max_workers=jobs or min(8, len(cmds))) as ex:
            list(ex.map(lambda c: _run(c, verbose), cmds))
        out_tmp = os.path.join(tmp, LIB_NAME)
        _run([cc, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", out_tmp], verbose)
        os.replace(out_tmp, LIB_PATH)
        with open(STAMP_PATH + ".tmp", "w") as f:
            f.write(stamp + "\n")
        os.replace(STAMP_PATH + ".tmp", STAMP_PATH)
    finally:
        shutil.rmtree(tmp, ignore_errors=True)
    return LIB_PATH


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
