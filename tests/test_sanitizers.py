"""The host controller under ThreadSanitizer and AddressSanitizer.

Sec. IV-C has the controller update the branch state atomically while
completion events of different agents arrive concurrently.  The controller,
C ABI and host models are built with -fsanitize=thread and with
-fsanitize=address (CPU only, recording executor) and exercised twice:
  * the native stress driver tests/native/abi_stress.cpp: events of every
    agent released from their own threads, racing duplicates, a thread
    polling branch states, infeasible frames and injected dispatch failures,
    in both release rules;
  * tests/test_abi.py and tests/test_checkpoint.py (the checkpoint parser
    on malformed files), with the sanitized host library and its runtime
    preloaded into the interpreter.
A sanitizer report, or a failed check, fails the test."""

import os
import subprocess
import sys

import pytest

import synth
from paper_2608_08330_amd import build_sanitize as BS
from paper_2608_08330_amd import rtcc as R

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SANITIZERS = ["thread", "address"]
REPORT = {"thread": "ThreadSanitizer", "address": "AddressSanitizer"}


@pytest.fixture(scope="module")
def model_files(tmp_path_factory):
    cfg = synth.config("t_attn")
    d = tmp_path_factory.mktemp("abi")
    desc, w = d / "desc.bin", d / "weights.bin"
    desc.write_bytes(bytes(R.model_desc(cfg)))
    w.write_bytes(R.weights_blob(cfg, synth.make_weights(cfg)).tobytes())
    return str(desc), str(w)


def _env(san, so):
    env = dict(os.environ)
    env["RTCC_HOSTTEST_LIB"] = so
    env["LD_PRELOAD"] = BS.runtime(san)
    env["TSAN_OPTIONS"] = "exitcode=66 halt_on_error=0"
    # the interpreter itself is not instrumented: its allocations are not
    # the library's leaks
    env["ASAN_OPTIONS"] = "detect_leaks=0 exitcode=66"
    return env


@pytest.mark.parametrize("san", SANITIZERS)
def test_stress_driver_is_clean(san, model_files):
    so, exe = BS.build(san)
    r = subprocess.run([exe, model_files[0], model_files[1], "300"], stdout=subprocess.PIPE,
                       stderr=subprocess.STDOUT, text=True, timeout=300)
    assert REPORT[san] not in r.stdout, r.stdout[-4000:]
    assert r.returncode == 0, r.stdout[-4000:]
    assert "300 frames ok" in r.stdout


@pytest.mark.parametrize("san", SANITIZERS)
def test_abi_tests_pass_under_sanitizer(san):
    so, _ = BS.build(san)
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-s", "-p", "no:cacheprovider", "-m", "not gpu",
                        "-k", "not library_loads", os.path.join(ROOT, "tests", "test_abi.py"),
                        os.path.join(ROOT, "tests", "test_checkpoint.py")],
                       stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True, timeout=600, cwd=ROOT,
                       env=_env(san, so))
    assert REPORT[san] not in r.stdout, r.stdout[-4000:]
    assert r.returncode == 0, r.stdout[-4000:]
