"""Sanitizer runs of the host code on the CPU: the host library (subgraph
build, redundancy reduction with its threaded pair counting, packing,
frontier sampling, induced subgraphs) under AddressSanitizer and
UndefinedBehaviorSanitizer, and the preparation pipeline's worker pool under
ThreadSanitizer. Each builds a small C++ driver (tests/sanitize/) against
the library's host sources with g++ and runs it; any sanitizer report fails
the test."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2001_02498_amd", "csrc")
HERE = os.path.join(ROOT, "tests", "sanitize")
GXX = shutil.which("g++")

pytestmark = pytest.mark.skipif(GXX is None, reason="g++ not found")


def _build(tmp_path, name, sanitize, sources, extra=()):
    exe = str(tmp_path / name)
    cmd = [GXX, "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer", "-pthread",
           f"-fsanitize={sanitize}", "-fno-sanitize-recover=all",
           f"-I{os.path.join(ROOT, 'include')}", f"-I{CSRC}"] + list(sources) + ["-o", exe]
    cmd += list(extra)
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, r.stderr[-4000:]
    return exe


def _run(exe, env_extra):
    env = dict(os.environ)
    env.update(env_extra)
    r = subprocess.run([exe], capture_output=True, text=True, timeout=900, env=env)
    report = r.stdout[-2000:] + r.stderr[-6000:]
    assert r.returncode == 0, report
    for marker in ("runtime error", "ERROR: AddressSanitizer", "WARNING: ThreadSanitizer",
                   "ERROR: LeakSanitizer"):
        assert marker not in r.stderr, report
    return r.stdout


def test_host_library_asan_ubsan(tmp_path):
    exe = _build(tmp_path, "host_harness", "address,undefined",
                 [os.path.join(HERE, "host_harness.cpp"), os.path.join(CSRC, "host_graph.cpp"),
                  os.path.join(CSRC, "sample.cpp")])
    out = _run(exe, {"ASAN_OPTIONS": "detect_leaks=1:halt_on_error=1",
                     "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1"})
    assert "0 failures" in out


def test_pipeline_tsan(tmp_path):
    # the pipeline source includes the HIP runtime header for its device
    # paths (pinned buffers, GPU-reducing workers), which host workers never
    # take; it is compiled as host C++ and linked against the HIP runtime
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    if not os.path.exists(os.path.join(rocm, "include", "hip", "hip_runtime.h")):
        pytest.skip("HIP headers not found")
    exe = _build(tmp_path, "pipeline_harness", "thread",
                 [os.path.join(HERE, "pipeline_harness.cpp"),
                  os.path.join(CSRC, "host_graph.cpp"), os.path.join(CSRC, "sample.cpp"),
                  "-x", "c++", os.path.join(CSRC, "pipeline.hip"), "-x", "none"],
                 extra=["-D__HIP_PLATFORM_AMD__", f"-I{rocm}/include", f"-L{rocm}/lib",
                        "-lamdhip64", f"-Wl,-rpath,{rocm}/lib"])
    out = _run(exe, {"TSAN_OPTIONS": "halt_on_error=1:second_deadlock_stack=1"})
    assert "0 failures" in out
