"""Compiles the HIP library in-tree for gfx950 (hipcc cross-compiles without a GPU)."""
from __future__ import annotations

import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
SOURCES = [os.path.join(CSRC, f) for f in
           ("host.hip", "host_plan.hip", "host_tables.hip", "host_next.hip", "host_check.cpp",
            "kern_general.hip", "kern_check.hip", "kern_pool.hip", "kern_sim.hip",
            "kern_greedy.hip", "kern_rollout.hip", "kern_costmodel.hip", "kern_memopt.hip",
            "kern_argmin.hip")]
LIB = os.path.join(HERE, "libdip_sim.so")
INCLUDE = os.path.join(ROOT, "include")

HIPCC_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared", "-Wall",
    # no packed fp32 instructions anywhere in the device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", "hipcc"):
        if cand and (os.path.sep not in cand or os.path.exists(cand)):
            return cand
    return "hipcc"


def build(jobs: int | None = None) -> str:
    """Each source to an object in parallel (the translation units share no
    device code), then one link into the shared library."""
    import concurrent.futures
    import tempfile

    cc = hipcc()
    compile_flags = [f for f in HIPCC_FLAGS if f != "-shared"]
    jobs = jobs or max(1, min(8, os.cpu_count() or 1))
    with tempfile.TemporaryDirectory(prefix="dip_sim_build_") as tmpdir:
        objs = [os.path.join(tmpdir, os.path.basename(src) + ".o") for src in SOURCES]

        def compile_one(src_obj):
            src, obj = src_obj
            subprocess.check_call([cc, *compile_flags, "-I", INCLUDE, "-I", CSRC, "-c", src,
                                   "-o", obj])

        with concurrent.futures.ThreadPoolExecutor(max_workers=jobs) as ex:
            list(ex.map(compile_one, zip(SOURCES, objs)))
        tmp = LIB + ".tmp"
        subprocess.check_call([cc, "--offload-arch=gfx950", "-fPIC", "-shared", "-o", tmp, *objs])
    os.replace(tmp, LIB)
    return LIB
