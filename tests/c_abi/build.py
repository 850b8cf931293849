"""Compile the plain-C caller of libgleam (detect.c) next to its source, against the
in-tree library; the C test runs the binary."""

from __future__ import annotations

import os
import shutil
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
BINARY = os.path.join(HERE, "detect")


def build() -> str:
    cc = shutil.which("gcc") or "gcc"
    cmd = [cc, "-std=c11", "-Wall", "-Wextra", "-Werror", "-O2", "-D__HIP_PLATFORM_AMD__",
           "-I/opt/rocm/include", "-I" + os.path.join(ROOT, "include"), os.path.join(HERE, "detect.c"),
           "-L" + os.path.join(ROOT, "paper_2607_23115_amd"), "-lgleam", "-L/opt/rocm/lib", "-lamdhip64",
           "-Wl,-rpath,$ORIGIN/../../paper_2607_23115_amd", "-Wl,-rpath,/opt/rocm/lib", "-o", BINARY]
    subprocess.run(cmd, check=True)
    return BINARY


if __name__ == "__main__":
    print(build())
