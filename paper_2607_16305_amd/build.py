"""Build liblookme.so (the C-ABI library and its gfx950 kernels) in-tree.

    python -m paper_2607_16305_amd.build [--jobs N] [--incremental]

Every source under csrc/ is compiled by hipcc for gfx950 only, then linked
into paper_2607_16305_amd/liblookme.so next to this file.
"""

from __future__ import annotations

import argparse
import concurrent.futures as cf
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "liblookme.so")
ROOT = os.path.dirname(HERE)

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

COMMON_FLAGS = [
    "-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
    # keep the compiler from forming packed fp32 ops (v_pk_fma_f32 and kin)
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function", "-Wno-unused-result",
    "-I", os.path.join(ROOT, "include"), "-I", CSRC,
]


def sources():
    return sorted(os.path.join(CSRC, f) for f in os.listdir(CSRC)
                  if f.endswith((".hip", ".cpp")))


def _inputs_key(src: str) -> str:
    """Hash of what an object depends on: the flags, the source and every
    header of the library (conservative: any header change rebuilds all)."""
    import hashlib
    h = hashlib.sha256(" ".join(COMMON_FLAGS).encode())
    for f in [src] + sorted(os.path.join(d, x) for d in (CSRC, os.path.join(ROOT, "include"))
                            for x in os.listdir(d) if x.endswith(".h")):
        with open(f, "rb") as fh:
            h.update(f.encode() + fh.read())
    return h.hexdigest()


def _compile(src: str, incremental: bool = False) -> str:
    obj = os.path.join(BUILD, os.path.basename(src) + ".o")
    key_file = obj + ".key"
    key = _inputs_key(src)
    if incremental and os.path.exists(obj) and os.path.exists(key_file):
        with open(key_file) as fh:
            if fh.read() == key:
                return obj
    cmd = [HIPCC, *COMMON_FLAGS, "-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    noise = "is not a recognized feature for this target"
    err = "\n".join(l for l in (r.stderr or "").splitlines() if noise not in l)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{err}")
    if err.strip():
        sys.stderr.write(err + "\n")
    with open(key_file, "w") as fh:
        fh.write(key)
    return obj


def build(jobs: int | None = None, incremental: bool = False) -> str:
    """Compile every source (or, with ``incremental``, only those whose
    inputs changed since their object was built) and link the library."""
    os.makedirs(BUILD, exist_ok=True)
    srcs = sources()
    jobs = jobs or min(len(srcs), max(1, (os.cpu_count() or 2) - 1))
    # the slowest source first, so that it does not start last
    srcs.sort(key=lambda f: -os.path.getsize(f))
    with cf.ThreadPoolExecutor(max_workers=jobs) as ex:
        objs = list(ex.map(lambda f: _compile(f, incremental), srcs))
    tmp = LIB + ".tmp"
    # -z defs: an unresolved symbol (say a kernel stub that was never
    # instantiated) fails the link instead of the first load
    cmd = [HIPCC, "-shared", "-fPIC", "-Wl,-z,defs", f"--offload-arch={ARCH}", *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stderr}")
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    ap = argparse.ArgumentParser()
    ap.add_argument("--jobs", type=int, default=None)
    ap.add_argument("--incremental", action="store_true",
                    help="recompile only sources whose inputs changed")
    args = ap.parse_args()
    print(build(args.jobs, args.incremental))
