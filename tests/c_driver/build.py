"""Build the plain-C driver of the C ABI (test infrastructure).

``tvl_c_driver`` uses only ``include/tvl.h`` and the HIP runtime, and links
the CPU oracle to check its results.  It is compiled with gcc as C99 next to
its source; the runtime paths of ``libtvl.so`` and ``liboracle.so`` are
recorded relative to the binary.
"""
from __future__ import annotations

import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
SRC = os.path.join(HERE, "tvl_c_driver.c")
BIN = os.path.join(HERE, "tvl_c_driver")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


def build() -> str:
    tmp = BIN + ".tmp%d" % os.getpid()
    cmd = ["gcc", "-std=c99", "-O2", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__",
           "-I", os.path.join(ROOT, "include"), "-I", os.path.join(ROCM, "include"), SRC,
           "-o", tmp, "-L", os.path.join(ROOT, "paper_2601_03324_amd"), "-ltvl",
           "-L", os.path.join(ROOT, "oracle"), "-loracle", "-L", os.path.join(ROCM, "lib"),
           "-lamdhip64", "-lm", "-Wl,-rpath,$ORIGIN/../../paper_2601_03324_amd",
           "-Wl,-rpath,$ORIGIN/../../oracle", "-Wl,-rpath," + os.path.join(ROCM, "lib")]
    subprocess.check_call(cmd)
    os.replace(tmp, BIN)
    return BIN


if __name__ == "__main__":
    print(build())
