"""Builds dip_client (a plain C caller of the library's C ABI) next to its
source, linked against the in-tree libdip_sim.so and the HIP runtime."""
from __future__ import annotations

import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
EXE = os.path.join(HERE, "dip_client")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


def build() -> str:
    lib_dir = os.path.join(ROOT, "paper_2504_14145_amd")
    rel = os.path.relpath(lib_dir, HERE)
    subprocess.check_call([
        "gcc", "-std=c11", "-O2", "-Wall", "-Wextra", "-D__HIP_PLATFORM_AMD__",
        "-I", os.path.join(ROOT, "include"), "-I", os.path.join(ROCM, "include"),
        os.path.join(HERE, "dip_client.c"), "-o", EXE + ".tmp",
        "-L", lib_dir, "-ldip_sim", "-L", os.path.join(ROCM, "lib"), "-lamdhip64",
        f"-Wl,-rpath,$ORIGIN/{rel}", f"-Wl,-rpath,{os.path.join(ROCM, 'lib')}",
    ])
    os.replace(EXE + ".tmp", EXE)
    return EXE


if __name__ == "__main__":
    print(build())
