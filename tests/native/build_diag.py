"""Builds the test-suite's diagnostic HIP library (tests/native/_build/libcham_diag.so) with
the library's own compiler flags, so the kernels under test compile as they do in the
library."""
from __future__ import annotations

import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
LIB = os.path.join(HERE, "_build", "libcham_diag.so")


def build() -> str:
    from paper_2609_33496_amd import build as libbuild
    os.makedirs(os.path.dirname(LIB), exist_ok=True)
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = [libbuild.HIPCC, *libbuild.FLAGS, "-shared", os.path.join(HERE, "cham_diag.hip"), "-o", tmp]
    subprocess.run(cmd, check=True, stdout=subprocess.PIPE, stderr=subprocess.STDOUT)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build())
