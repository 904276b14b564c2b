"""Build the plain C-ABI consumer test (tests/c/abi_forward.cpp).

A host-only C++ program: it includes include/bitlogic.h, links the product
library (paper_2602_07400_amd/libbitlogic.so) and the CPU oracle
(oracle/liboracle.so), and finds both at run time through an $ORIGIN-relative
rpath, so the built binary works from any copy of the tree.  Called by
__graft_entry__.build(); tests/test_c_abi_gpu.py runs the result.
"""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
SRC = os.path.join(HERE, "abi_forward.cpp")
EXE = os.path.join(HERE, "abi_forward")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


def build() -> str:
    """Compile and link the consumer; needs libbitlogic.so and liboracle.so built."""
    for lib in ("paper_2602_07400_amd/libbitlogic.so", "oracle/liboracle.so"):
        if not os.path.exists(os.path.join(ROOT, lib)):
            raise RuntimeError(f"{lib} is not built")
    tmp = EXE + ".tmp%d" % os.getpid()
    cmd = ["g++", "-O2", "-std=c++17", "-Wall", "-D__HIP_PLATFORM_AMD__",
           "-I", os.path.join(ROOT, "include"), "-I", os.path.join(ROCM, "include"),
           SRC, "-o", tmp,
           "-L", os.path.join(ROOT, "paper_2602_07400_amd"), "-L", os.path.join(ROOT, "oracle"),
           "-L", os.path.join(ROCM, "lib"), "-lbitlogic", "-loracle", "-lamdhip64",
           "-Wl,-rpath,$ORIGIN/../../paper_2602_07400_amd:$ORIGIN/../../oracle:"
           + os.path.join(ROCM, "lib")]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"building the C-ABI test failed:\n{r.stderr}")
    os.replace(tmp, EXE)
    return EXE


if __name__ == "__main__":
    print(build())
    sys.exit(0)
