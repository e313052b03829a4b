"""The host side of the C ABI under AddressSanitizer (CPU only).

Builds a variant of the library whose host ABI code (lookme_abi.cpp:
argument validation, workspace layout, handle bookkeeping) is compiled with
AddressSanitizer, links it with the device objects of the normal in-tree
build, and runs tests/test_abi_cpu.py against it in a child process with the
sanitizer runtime preloaded.  Only host code is instrumented (the sanitizer
flag goes to the host compilation only); no GPU is used.
"""

import glob
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2607_16305_amd")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


def _asan_runtime():
    hits = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    return hits[-1] if hits else None


def test_abi_validation_under_address_sanitizer(tmp_path):
    objs = [o for o in sorted(glob.glob(os.path.join(PKG, "_build", "*.o")))
            if not os.path.basename(o).startswith("lookme_abi")]
    rt = _asan_runtime()
    if not os.path.exists(HIPCC) or rt is None or not objs:
        pytest.skip("needs hipcc, the clang sanitizer runtime and a built library (build())")
    abi = os.path.join(tmp_path, "lookme_abi.o")
    lib = os.path.join(tmp_path, "liblookme_asan.so")
    host_asan = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fno-omit-frame-pointer"]
    subprocess.run([HIPCC, "-O1", "-g", "-std=c++17", "-fPIC", "--offload-arch=gfx950",
                    *host_asan, "-I", os.path.join(ROOT, "include"),
                    "-I", os.path.join(PKG, "csrc"), "-c",
                    os.path.join(PKG, "csrc", "lookme_abi.cpp"), "-o", abi],
                   check=True, capture_output=True)
    subprocess.run([HIPCC, "-shared", "-fPIC", "--offload-arch=gfx950",
                    "-Xarch_host", "-fsanitize=address", abi, *objs, "-o", lib],
                   check=True, capture_output=True)
    code = ("import sys; sys.path.insert(0, %r); "
            "import paper_2607_16305_amd.lookme as lk; lk.LIB_PATH = %r; "
            "import pytest; sys.exit(pytest.main(['-q', '-p', 'no:cacheprovider', %r]))"
            % (ROOT, lib, os.path.join(ROOT, "tests", "test_abi_cpu.py")))
    env = dict(os.environ, LD_PRELOAD=rt, ASAN_OPTIONS="detect_leaks=0:halt_on_error=1")
    r = subprocess.run([sys.executable, "-c", code], env=env, capture_output=True, text=True,
                       timeout=600, cwd=ROOT)
    out = r.stdout + r.stderr
    assert "AddressSanitizer" not in out, out[-4000:]
    assert r.returncode == 0, out[-4000:]
    assert " passed" in out
