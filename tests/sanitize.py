"""Run the CPU test suite against sanitizer builds of the host code.

Builds, in a scratch copy of the tree, the product library with its host code
(the C-ABI argument checks, workspace planning, table specialization) under
AddressSanitizer and UndefinedBehaviorSanitizer, and the CPU oracle under the
same sanitizers, then runs ``pytest -m "not gpu"`` there with the sanitizer
runtime preloaded.  Device code is compiled as usual; no GPU is needed.

    python tests/sanitize.py            # prints the pytest summary; exit status is pytest's

Both libraries are built with ROCm's clang so that one sanitizer runtime
serves the whole process.  Leak checking is off: the Python interpreter
itself does not free everything at exit.
"""
from __future__ import annotations

import glob
import os
import shutil
import subprocess
import sys
import tempfile

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
LLVM = os.path.join(ROCM, "llvm", "bin")
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer",
       "-g"]


def _runtime() -> str:
    hits = glob.glob(os.path.join(ROCM, "llvm", "lib", "clang", "*", "lib", "linux",
                                  "libclang_rt.asan-x86_64.so"))
    if not hits:
        raise RuntimeError("clang's shared AddressSanitizer runtime was not found")
    return hits[0]


def _copy_tree(dst: str) -> None:
    ignore = shutil.ignore_patterns("_build", "__pycache__", "*.so", "*.o", "abi_forward",
                                    ".pytest_cache")
    for name in ("paper_2602_07400_amd", "include", "oracle", "tests"):
        shutil.copytree(os.path.join(ROOT, name), os.path.join(dst, name), ignore=ignore)
    for name in ("__graft_entry__.py", "bench.py"):
        shutil.copy(os.path.join(ROOT, name), dst)


def _build_library(tree: str) -> None:
    sys.path.insert(0, tree)
    from paper_2602_07400_amd import build as B        # the copy's build settings
    objs = []
    os.makedirs(os.path.join(tree, "_sanobj"))
    host_san = [f for flag in SAN for f in ("-Xarch_host", flag)]
    for src in B.SOURCES:
        obj = os.path.join(tree, "_sanobj", src.replace(".hip", ".o"))
        cmd = [B.hipcc(), *B.HIPCC_FLAGS, *host_san, "-I", os.path.join(tree, "include"), "-c",
               os.path.join(tree, "paper_2602_07400_amd", "csrc", src), "-o", obj]
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError(f"hipcc failed on {src}:\n{r.stderr}")
        objs.append(obj)
    lib = os.path.join(tree, "paper_2602_07400_amd", "libbitlogic.so")
    subprocess.run([os.path.join(LLVM, "clang++"), "-shared", "-shared-libsan", *SAN, "-o", lib,
                    *objs, "-L", os.path.join(ROCM, "lib"), "-lamdhip64",
                    "-Wl,-rpath," + os.path.join(ROCM, "lib")], check=True)


def _build_oracle(tree: str) -> None:
    src = os.path.join(tree, "oracle", "bitlogic_oracle.c")
    lib = os.path.join(tree, "oracle", "liboracle.so")
    subprocess.run([os.path.join(LLVM, "clang"), "-O1", "-fopenmp", "-shared", "-fPIC",
                    "-shared-libsan", *SAN, "-o", lib, src,
                    "-Wl,-rpath," + os.path.join(ROCM, "llvm", "lib")], check=True)


def main() -> int:
    rt = _runtime()
    with tempfile.TemporaryDirectory(prefix="bitlogic_san_") as tree:
        _copy_tree(tree)
        _build_library(tree)
        _build_oracle(tree)
        env = dict(os.environ)
        env["LD_PRELOAD"] = rt
        env["ASAN_OPTIONS"] = "detect_leaks=0:halt_on_error=1:abort_on_error=1"
        env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1"
        env["PYTHONDONTWRITEBYTECODE"] = "1"
        # the plain C++ consumer links the libraries with g++, which lacks the
        # sanitizer runtime the instrumented libraries need; it is built and
        # run against the normal build by the regular suite
        r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-m", "not gpu",
                            "-p", "no:cacheprovider", "--deselect",
                            "tests/test_c_abi_gpu.py::test_c_consumer_builds_against_header",
                            "tests"], cwd=tree, env=env)
        return r.returncode


if __name__ == "__main__":
    sys.exit(main())
