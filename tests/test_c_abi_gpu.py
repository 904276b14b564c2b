"""A plain C++ program drives the library through include/bitlogic.h alone.

tests/c/abi_forward.cpp allocates with the HIP runtime, runs bitlogic_forward
(thermometer encoder, GroupSum head) and bitlogic_network_forward (binary
encoder, quantized head) on 3 * 1024 + 37 samples, and compares scores,
logits and argmax with the CPU oracle's C entry points element by element;
it also checks that a NULL input is rejected with BITLOGIC_ERR_NULL before
anything is enqueued.  No Python binding is involved.
"""
import importlib.util
import os
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
EXE = os.path.join(HERE, "c", "abi_forward")


def _exe() -> str:
    if not os.path.exists(EXE):
        spec = importlib.util.spec_from_file_location("c_abi_build",
                                                      os.path.join(HERE, "c", "build.py"))
        mod = importlib.util.module_from_spec(spec)
        spec.loader.exec_module(mod)
        mod.build()
    return EXE


def test_c_consumer_builds_against_header():
    # host only: the program compiles and links against the header and both libraries
    assert os.access(_exe(), os.X_OK)


@pytest.mark.gpu
def test_c_consumer_forward_matches_oracle():
    print("[c abi] running", EXE, flush=True)
    r = subprocess.run([_exe()], capture_output=True, text=True, timeout=120)
    print(r.stdout, r.stderr, flush=True)
    assert r.returncode == 0, f"exit {r.returncode}: {r.stdout}\n{r.stderr}"
    assert "c abi ok" in r.stdout
