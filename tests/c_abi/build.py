"""Compile the plain-C callers of libgleam (detect.c, remap.c) next to their sources,
against the in-tree library; the C tests run the binaries."""

from __future__ import annotations

import os
import shutil
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
PROGRAMS = ("detect", "remap")


def build() -> list[str]:
    cc = shutil.which("gcc") or "gcc"
    out = []
    for name in PROGRAMS:
        binary = os.path.join(HERE, name)
        cmd = [cc, "-std=c11", "-Wall", "-Wextra", "-Werror", "-O2", "-D__HIP_PLATFORM_AMD__",
               "-I/opt/rocm/include", "-I" + os.path.join(ROOT, "include"), os.path.join(HERE, name + ".c"),
               "-L" + os.path.join(ROOT, "paper_2607_23115_amd"), "-lgleam", "-L/opt/rocm/lib", "-lamdhip64",
               "-Wl,-rpath,$ORIGIN/../../paper_2607_23115_amd", "-Wl,-rpath,/opt/rocm/lib", "-o", binary]
        subprocess.run(cmd, check=True)
        out.append(binary)
    return out


if __name__ == "__main__":
    print(build())
