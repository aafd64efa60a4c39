"""Build tests/native/_build/abi_driver_asan: the C-ABI driver (abi_driver.cpp)
linked with the library's sources, AddressSanitizer on the host code only
(`-Xarch_host` before each sanitizer flag: the device code is built as in the
library).  Run the executable on a machine with a GPU, with leak detection
and the ROCm runtime's own allocations suppressed:

  ASAN_OPTIONS=detect_leaks=1 \
  LSAN_OPTIONS=suppressions=tests/native/lsan_rocm_runtime.supp \
  tests/native/_build/abi_driver_asan

It prints one line per call and "abi driver ok".  Not part of the library
build."""
from __future__ import annotations

import os
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

from paper_2108_03917_amd import _build as B  # noqa: E402

OUT = os.path.join(HERE, "_build")
EXE = os.path.join(OUT, "abi_driver_asan")
HOST_ASAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fno-omit-frame-pointer", "-g"]


def build() -> str:
    os.makedirs(OUT, exist_ok=True)
    jobs, objs = [], []
    for src in B.SOURCES:
        obj = os.path.join(OUT, src.replace(".hip", ".o"))
        objs.append(obj)
        jobs.append([B.hipcc(), *B.common_flags(), *B.EXTRA.get(src, []), *HOST_ASAN, "-c",
                     os.path.join(B.CSRC, src), "-o", obj])
    drv = os.path.join(OUT, "abi_driver.o")
    objs.append(drv)
    jobs.append([B.hipcc(), *B.common_flags(), *HOST_ASAN, "-x", "hip", "-c", os.path.join(HERE, "abi_driver.cpp"),
                 "-o", drv])
    with ThreadPoolExecutor(max_workers=8) as ex:
        list(ex.map(B._run, jobs))
    B._run([B.hipcc(), f"--offload-arch={B.ARCH}", *HOST_ASAN, *objs, "-o", EXE])
    return EXE


if __name__ == "__main__":
    print(build())
