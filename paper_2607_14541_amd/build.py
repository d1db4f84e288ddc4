"""Build the gfx950 shared library libatrex.so (C ABI in include/atrex.h) and
the host-side synthetic trace generator, in-tree.

    python -m paper_2607_14541_amd.build
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libatrex.so")
# plain 1 GiB copy, the known-size kernel the HBM byte counters are scaled by
COPY_CAL = os.path.join(HERE, "copy_calibration")
BUILD_DIR = os.path.join(HERE, "_build")

HIP_SOURCES = ["atrex_host.hip", "kernels_aggregate.hip", "kernels_rows.hip", "kernels_util.hip",
               "kernels_normalize.hip", "kernels_small.hip", "kernels_units.hip", "kernels_score.hip",
               "kernels_share.hip", "kernels_stats.hip", "kernels_join.hip"]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
HIP_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-fPIC", "-std=c++17",
    # no packed fp32 instructions (v_pk_*_f32) anywhere in the library
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # no contraction: the fp64 score must be the plain product and sum
    "-ffp-contract=off",
    "-Wall", "-Wno-unused-command-line-argument",
    "-I" + os.path.join(ROOT, "include"),
]


def _compile(src: str) -> str:
    obj = os.path.join(BUILD_DIR, os.path.splitext(src)[0] + ".o")
    cmd = [HIPCC, *HIP_FLAGS, "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(r.stdout + r.stderr)
        raise RuntimeError("hipcc failed on " + src)
    return obj


def build_lib() -> str:
    os.makedirs(BUILD_DIR, exist_ok=True)
    with cf.ThreadPoolExecutor(max_workers=4) as ex:
        objs = list(ex.map(_compile, HIP_SOURCES))
    tmp = LIB + ".tmp%d" % os.getpid()
    subprocess.check_call([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp, *objs])
    os.replace(tmp, LIB)
    return LIB


def build_copy_calibration() -> str:
    tmp = COPY_CAL + ".tmp%d" % os.getpid()
    subprocess.check_call([HIPCC, *HIP_FLAGS, "-o", tmp, os.path.join(CSRC, "copy_calibration.hip")])
    os.replace(tmp, COPY_CAL)
    return COPY_CAL


def build_all() -> None:
    from . import synth
    build_lib()
    build_copy_calibration()
    synth.build(force=True)


if __name__ == "__main__":
    build_all()
    print("built", LIB)
