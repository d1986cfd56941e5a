"""Build the native libraries in-tree.

  lib/librtcc.so           the gfx950 library (HIP kernels + C ABI)
  lib/librtcc_hosttest.so  the same controller and C ABI linked against a
                           recording executor, for host-only tests

Usage: python -m paper_2608_08330_amd.build [--jobs N] [--only gpu|host]
"""

import argparse
import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "lib")
OBJ = os.path.join(HERE, "_build")
ROOT = os.path.dirname(HERE)
INCLUDE = os.path.join(ROOT, "include")

ARCH = "gfx950"
HIPCC = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
CXX = shutil.which("g++") or "g++"

HOST_SOURCES = ["api.cpp", "checkpoint.cpp", "controller.cpp", "model.cpp", "uplink.cpp", "kernels/conv_plan.cpp"]
HIP_SOURCES = [
    "executor_hip.hip",
    "kernels/pillar.hip",
    "kernels/igemm.hip",
    "kernels/post.hip",
    "kernels/nms.hip",
    "nms_api.hip",
    "nms_noalloc.hip",
]

# Packed fp32 instructions are disabled for every device compile.
HIP_FLAGS = [
    "-O3", "-std=c++17", "-fPIC", "--offload-arch=" + ARCH,
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-result", "-fvisibility=hidden", "-I" + INCLUDE,
]
# Host code never contracts a * b + c into an FMA, so its floating point
# follows the written order of operations.
HOST_FLAGS = ["-O2", "-std=c++17", "-fPIC", "-Wall", "-Wextra", "-ffp-contract=off", "-fvisibility=hidden",
              "-I" + INCLUDE]


def _run(cmd):
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    if r.returncode != 0:
        raise RuntimeError("build step failed:\n%s\n%s" % (" ".join(cmd), r.stdout))
    return r.stdout


def _obj(src, tag):
    return os.path.join(OBJ, tag, src.replace("/", "_") + ".o")


def build_gpu(jobs):
    os.makedirs(os.path.join(OBJ, "gpu"), exist_ok=True)
    os.makedirs(LIB, exist_ok=True)
    cmds = []
    for s in HOST_SOURCES:
        cmds.append([CXX] + HOST_FLAGS + ["-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include", "-c",
                                          os.path.join(CSRC, s), "-o", _obj(s, "gpu")])
    for s in HIP_SOURCES:
        cmds.append([HIPCC] + HIP_FLAGS + ["-c", os.path.join(CSRC, s), "-o", _obj(s, "gpu")])
    with ThreadPoolExecutor(max_workers=jobs) as ex:
        list(ex.map(_run, cmds))
    out = os.path.join(LIB, "librtcc.so")
    tmp = out + ".tmp"
    _run([HIPCC, "-shared", "-fPIC", "--offload-arch=" + ARCH, "-o", tmp]
         + [_obj(s, "gpu") for s in HOST_SOURCES + HIP_SOURCES])
    os.replace(tmp, out)
    return out


def build_host(jobs):
    os.makedirs(os.path.join(OBJ, "host"), exist_ok=True)
    os.makedirs(LIB, exist_ok=True)
    srcs = HOST_SOURCES + ["fake_executor.cpp"]
    cmds = [[CXX] + HOST_FLAGS + ["-g", "-c", os.path.join(CSRC, s), "-o", _obj(s, "host")] for s in srcs]
    with ThreadPoolExecutor(max_workers=jobs) as ex:
        list(ex.map(_run, cmds))
    out = os.path.join(LIB, "librtcc_hosttest.so")
    tmp = out + ".tmp"
    _run([CXX, "-shared", "-fPIC", "-o", tmp] + [_obj(s, "host") for s in srcs] + ["-lpthread"])
    os.replace(tmp, out)
    return out


def build(jobs=8, only=None):
    outs = []
    if only in (None, "host"):
        outs.append(build_host(jobs))
    if only in (None, "gpu"):
        outs.append(build_gpu(jobs))
    return outs


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--jobs", type=int, default=min(8, os.cpu_count() or 1))
    ap.add_argument("--only", choices=["gpu", "host"])
    a = ap.parse_args(argv)
    for o in build(a.jobs, a.only):
        print(o)


if __name__ == "__main__":
    sys.exit(main())
