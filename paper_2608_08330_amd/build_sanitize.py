"""Sanitizer builds of the host-side controller (CPU only, no device code).

The controller, C ABI, model checks and uplink models are compiled with g++
and -fsanitize=thread or -fsanitize=address and linked against the recording
executor, both as a shared library (lib/librtcc_hosttest_<san>.so, loadable
with the sanitizer runtime preloaded) and as the native stress driver
tests/native/abi_stress.cpp (bin/abi_stress_<san>).

Usage: python -m paper_2608_08330_amd.build_sanitize {thread,address}
"""

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

from paper_2608_08330_amd.build import CSRC, CXX, HOST_SOURCES, INCLUDE, LIB, OBJ, ROOT

SOURCES = HOST_SOURCES + ["fake_executor.cpp"]
DRIVER = os.path.join(ROOT, "tests", "native", "abi_stress.cpp")
BIN = os.path.join(os.path.dirname(LIB), "bin")


def _flags(san):
    return ["-O1", "-g", "-std=c++17", "-fPIC", "-Wall", "-ffp-contract=off", "-fno-omit-frame-pointer",
            "-fsanitize=" + san, "-I" + INCLUDE]


def _run(cmd):
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    if r.returncode != 0:
        raise RuntimeError("build step failed:\n%s\n%s" % (" ".join(cmd), r.stdout))


def build(san, jobs=8):
    """Returns (shared library, stress driver) paths."""
    if san not in ("thread", "address"):
        raise ValueError(san)
    odir = os.path.join(OBJ, "san_" + san)
    os.makedirs(odir, exist_ok=True)
    os.makedirs(LIB, exist_ok=True)
    os.makedirs(BIN, exist_ok=True)
    objs = [os.path.join(odir, s.replace("/", "_") + ".o") for s in SOURCES]
    cmds = [[CXX] + _flags(san) + ["-c", os.path.join(CSRC, s), "-o", o] for s, o in zip(SOURCES, objs)]
    with ThreadPoolExecutor(max_workers=jobs) as ex:
        list(ex.map(_run, cmds))
    so = os.path.join(LIB, "librtcc_hosttest_%s.so" % san)
    _run([CXX, "-shared", "-fsanitize=" + san, "-o", so] + objs + ["-lpthread"])
    exe = os.path.join(BIN, "abi_stress_%s" % san)
    _run([CXX] + _flags(san) + ["-o", exe, DRIVER] + objs + ["-lpthread"])
    return so, exe


def runtime(san):
    """Path of the sanitizer runtime to preload into an uninstrumented host."""
    lib = {"thread": "libtsan.so", "address": "libasan.so"}[san]
    return subprocess.run([CXX, "-print-file-name=" + lib], stdout=subprocess.PIPE, text=True,
                          check=True).stdout.strip()


if __name__ == "__main__":
    for p in build(sys.argv[1]):
        print(p)
