"""The CPU oracle (oracle/gs_oracle.c) and the host planner
(paper_2607_19893_amd/csrc/planner.cpp) under AddressSanitizer and
UndefinedBehaviorSanitizer: host code only, built here with gcc / g++.

  * the oracle's shared library, built with both sanitizers, is loaded by a
    child Python process (the sanitizer runtime preloaded, leak checks off
    for the interpreter) that runs one training view, a task unit, renders
    with planted mistakes and the SH helpers (tests/sanitize/oracle_run.py);
  * the planner, built with both sanitizers into a small driver
    (tests/sanitize/planner_driver.cpp, leak checks on), builds graphs,
    partitions and schedules of seeded captures (one large enough for the
    threaded graph build) and refuses malformed inputs; its digest of every
    result must equal that of a plain build of the same sources.

Any report from either sanitizer stops the run (halt on error) and fails
the test.
"""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HERE = os.path.dirname(os.path.abspath(__file__))
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-g", "-O1"]

pytestmark = pytest.mark.skipif(shutil.which("gcc") is None or shutil.which("g++") is None,
                                reason="needs gcc and g++")


def _runtime(name):
    p = subprocess.check_output(["gcc", "-print-file-name=" + name], text=True).strip()
    if not os.path.isabs(p) or not os.path.exists(p):
        pytest.skip("no %s for this gcc" % name)
    return p


def _env(**kw):
    env = dict(os.environ)
    env.update(kw)
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1"
    env["OMP_NUM_THREADS"] = "4"
    return env


def _no_reports(r):
    text = r.stdout + r.stderr
    assert r.returncode == 0 and "runtime error" not in text and "AddressSanitizer" not in text, text[-4000:]


def test_planner_under_sanitizers(tmp_path):
    srcs = [os.path.join(ROOT, "paper_2607_19893_amd", "csrc", "planner.cpp"),
            os.path.join(HERE, "sanitize", "planner_driver.cpp")]
    inc = ["-I" + os.path.join(ROOT, "include"), "-I" + os.path.join(ROOT, "paper_2607_19893_amd", "csrc")]
    common = ["g++", "-std=c++17", "-ffp-contract=off", "-pthread"] + inc
    san, plain = str(tmp_path / "planner_san"), str(tmp_path / "planner_plain")
    subprocess.check_call(common + SAN + srcs + ["-o", san])
    subprocess.check_call(common + ["-O2"] + srcs + ["-o", plain])
    r = subprocess.run([san], capture_output=True, text=True, timeout=300,
                       env=_env(ASAN_OPTIONS="detect_leaks=1:halt_on_error=1"))
    _no_reports(r)
    p = subprocess.run([plain], capture_output=True, text=True, timeout=300)
    assert p.returncode == 0 and r.stdout.strip() == p.stdout.strip() and r.stdout.startswith("digest")


def test_oracle_under_sanitizers(tmp_path):
    lib = str(tmp_path / "liborc_san.so")
    subprocess.check_call(["gcc", "-std=gnu11", "-fopenmp", "-ffp-contract=off", "-fno-fast-math", "-fPIC",
                           "-shared"] + SAN + [os.path.join(ROOT, "oracle", "gs_oracle.c"), "-o", lib, "-lm"])
    syms = subprocess.check_output(["nm", "-D", "--undefined-only", lib], text=True)
    assert "__asan_" in syms and "__ubsan_" in syms          # the library is instrumented
    env = _env(GS_ORACLE_LIB=lib, LD_PRELOAD=_runtime("libasan.so"),
               ASAN_OPTIONS="detect_leaks=0:halt_on_error=1:verify_asan_link_order=0")
    r = subprocess.run([sys.executable, os.path.join(HERE, "sanitize", "oracle_run.py")], capture_output=True,
                       text=True, timeout=600, env=env, cwd=ROOT)
    _no_reports(r)
    assert r.stdout.strip().endswith("ok")
