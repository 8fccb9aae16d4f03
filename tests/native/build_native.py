"""Build the host-sanitizer copy of the library and its C ABI driver.

The library sources are compiled as for the product (same hipcc flags, gfx950
kernels) with AddressSanitizer and UndefinedBehaviorSanitizer on the host side
only (each -fsanitize= after -Xarch_host: the GPU code is built as usual), and
linked as tests/native/_out/libwdc_hostsan.so. The C99 driver abi_driver.c is
compiled with the same sanitizers (its runtime serves the library too) into
tests/native/_out/abi_driver. Outputs are rebuilt on every call.

Usage: python tests/native/build_native.py  (also run by __graft_entry__.build()).
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
OUT = os.path.join(HERE, "_out")
LIB = os.path.join(OUT, "libwdc_hostsan.so")
DRIVER = os.path.join(OUT, "abi_driver")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
CLANG = os.path.join(ROCM, "llvm", "bin", "clang")

HOST_SAN = ["-g", "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer"]


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"{' '.join(cmd[:3])} ... failed:\n{r.stderr[-4000:]}")


def build(verbose: bool = False) -> str:
    sys.path.insert(0, ROOT)
    from paper_2608_01845_amd import build as pb
    os.makedirs(os.path.join(OUT, "obj"), exist_ok=True)

    def compile_one(src):
        obj = os.path.join(OUT, "obj", os.path.splitext(src)[0] + ".o")
        _run([pb.HIPCC, *pb.FLAGS, *HOST_SAN, "-c", os.path.join(pb.CSRC, src), "-o", obj])
        return obj

    with ThreadPoolExecutor(max_workers=min(len(pb.SOURCES), 8)) as ex:
        objs = list(ex.map(compile_one, pb.SOURCES))
    _run([pb.HIPCC, "-shared", "-fPIC", f"--offload-arch={pb.ARCH}", *objs, "-o", LIB + ".tmp"])
    os.replace(LIB + ".tmp", LIB)
    clang = CLANG if os.path.exists(CLANG) else (shutil.which("clang") or CLANG)
    _run([clang, "-std=c99", "-g", "-O1", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__",
          f"-I{ROCM}/include", f"-I{os.path.join(ROOT, 'include')}",
          "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer",
          os.path.join(HERE, "abi_driver.c"), "-o", DRIVER + ".tmp",
          f"-L{OUT}", "-lwdc_hostsan", f"-L{ROCM}/lib", "-lamdhip64", "-lm",
          "-Wl,-rpath,$ORIGIN", f"-Wl,-rpath,{ROCM}/lib"])
    os.replace(DRIVER + ".tmp", DRIVER)
    if verbose:
        print("built", LIB, "and", DRIVER)
    return DRIVER


if __name__ == "__main__":
    build(verbose=True)
