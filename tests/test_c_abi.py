"""The C ABI driven from a plain C program (tests/c/kap_c_smoke.c, built by
__graft_entry__.build() with gcc against include/kap.h and the HIP runtime):
host-side validation without a GPU, and on the GPU the worked plan vector in
page and token mode under both policies plus the one-visible-token closed
form of decode and verify."""
import os
import subprocess

import pytest

BIN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "c", "kap_c_smoke")


def run(mode):
    if not os.path.exists(BIN):
        pytest.fail("tests/c/kap_c_smoke is not built; run __graft_entry__.build() first")
    r = subprocess.run([BIN, mode], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0 and "PASSED" in r.stdout, r.stdout + r.stderr
    return r.stdout


def test_c_program_validation():
    out = run("cpu")
    assert "ok cpu checks" in out


@pytest.mark.gpu
def test_c_program_on_the_gpu():
    out = run("gpu")
    assert out.count("ok plan vector") == 4 and out.count("ok one visible token") == 3
    assert "ok one visible token (scheduled decode)" in out
