"""Builds libseedq.so (HIP for gfx950 + host C++) in place, next to this file."""
from __future__ import annotations

import os
import subprocess
import sys
import tempfile

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB_NAME = "libseedq.so"
LIB_PATH = os.path.join(HERE, LIB_NAME)

HIP_SOURCES = ["seedq_bases.hip", "seedq_search_mfma.hip", "seedq_compact.hip",
               "seedq_decompress.hip", "seedq_stream.hip",
               "seedq_footprint.hip", "seedq_frontend.hip", "seedq_noalloc.hip"]
HOST_SOURCES = ["seedq_api.cpp", "seedq_schedule.cpp", "seedq_frontend_host.cpp"]

# Device code is compiled without packed fp32 instructions.
DEVICE_FLAGS = ["--offload-arch=gfx950", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
                "-mllvm", "-amdgpu-mfma-vgpr-form"]
COMMON = ["-O3", "-std=c++17", "-fPIC", "-I" + INCLUDE, "-I" + CSRC, "-Wall", "-Wno-unused-function"]


def hipcc() -> str:
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    return os.path.join(rocm, "bin", "hipcc")


def build(verbose: bool = False, jobs: int = 8) -> str:
    """Compile every source and link libseedq.so; returns its path."""
    with tempfile.TemporaryDirectory(prefix="seedq_build_") as tmp:
        procs, objs = [], []
        for src in HIP_SOURCES:
            obj = os.path.join(tmp, src + ".o")
            cmd = [hipcc(), "-x", "hip", *DEVICE_FLAGS, *COMMON, "-c", os.path.join(CSRC, src), "-o", obj]
            procs.append((cmd, subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT)))
            objs.append(obj)
        for src in HOST_SOURCES:
            obj = os.path.join(tmp, src + ".o")
            # host-only translation units; no fused multiply-add in the planner's fp64
            cmd = [hipcc(), *COMMON, "-ffp-contract=off", "-D__HIP_PLATFORM_AMD__", "-c",
                   os.path.join(CSRC, src), "-o", obj]
            procs.append((cmd, subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT)))
            objs.append(obj)
        failed = []
        for cmd, p in procs:
            out, _ = p.communicate()
            text = out.decode(errors="replace")
            if p.returncode != 0:
                failed.append((cmd, text))
            elif verbose and text.strip():
                print(text, file=sys.stderr)
        if failed:
            msg = "\n\n".join(" ".join(c) + "\n" + t for c, t in failed)
            raise RuntimeError("libseedq build failed:\n" + msg)
        tmp_lib = LIB_PATH + ".tmp"
        link = [hipcc(), *DEVICE_FLAGS, "-shared", "-fPIC", *objs, "-o", tmp_lib]
        subprocess.run(link, check=True)
        os.replace(tmp_lib, LIB_PATH)
    return LIB_PATH


if __name__ == "__main__":
    print(build(verbose=True))
