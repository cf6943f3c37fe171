"""Host-sanitized build of libsgemm_emu.so, for CPU checks of the C ABI.

Every translation unit is compiled as in build.py, with AddressSanitizer and
UndefinedBehaviorSanitizer applied to the host pass only (the device code is
the same gfx950 code as in the product build).  The library is written to
_build/sanitize/libsgemm_emu.so; load it with SGEMM_EMU_LIB pointing at it
and clang's ASan runtime preloaded (``asan_runtime()``).  It is a checking
build for hosts without a GPU: the argument validation, extent arithmetic,
policy resolution and host-mirrored index maps run under the sanitizers.

    python paper_2308_15152_amd/build_sanitized.py
"""
from __future__ import annotations

import concurrent.futures as cf
import glob
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, HERE)
import build as product  # noqa: E402

OUT_DIR = os.path.join(product.ROOT, "_build", "sanitize")
LIB_PATH = os.path.join(OUT_DIR, product.LIB_NAME)

HOST_SANITIZE = ["-Xarch_host", "-fsanitize=address,undefined",
                 "-Xarch_host", "-fno-sanitize-recover=all",
                 "-Xarch_host", "-fno-omit-frame-pointer"]


def asan_runtime() -> str:
    """clang's ASan runtime shared library (the one the host pass links)."""
    llvm = os.path.dirname(os.path.dirname(os.path.realpath(product.HIPCC)))
    for cand in sorted(glob.glob(os.path.join(
            llvm, "llvm", "lib", "clang", "*", "lib", "linux", "libclang_rt.asan-x86_64.so"))):
        return cand
    for cand in sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/"
                                 "libclang_rt.asan-x86_64.so")):
        return cand
    raise FileNotFoundError("clang ASan runtime not found")


def _compile(src: str) -> str:
    obj = os.path.join(OUT_DIR, os.path.basename(src) + ".o")
    cmd = [product.HIPCC, *product.DEVICE_FLAGS, *HOST_SANITIZE, "-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed on {src}:\n{r.stderr[-4000:]}")
    return obj


def build() -> str:
    os.makedirs(OUT_DIR, exist_ok=True)
    srcs = product.sources()
    with cf.ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        objs = list(ex.map(_compile, srcs))
    tmp = LIB_PATH + ".tmp"
    subprocess.run([product.HIPCC, f"--offload-arch={product.ARCH}", "-shared", "-fPIC",
                    *HOST_SANITIZE, *objs, "-o", tmp], check=True)
    os.replace(tmp, LIB_PATH)
    return LIB_PATH


if __name__ == "__main__":
    print(build())
