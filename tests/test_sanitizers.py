"""The host code under the host compiler's sanitizers (CPU only).

- The host half of libvie (api.cpp, builder.cpp, index_io.cpp) is built with
  g++ and AddressSanitizer + UndefinedBehaviorSanitizer (leak checks on),
  and again with ThreadSanitizer, against stand-ins for the kernels and the
  HIP runtime (tests/sanitize/device_stubs.cpp), and driven through the C
  ABI by tests/sanitize/host_driver.cpp: the multithreaded builder, the
  index file with corrupt and truncated copies, export, and the error paths,
  among them an allocation failure that must give VIE_ENOMEM without a leak.
- The oracle (oracle/oracle.c) is built with AddressSanitizer +
  UndefinedBehaviorSanitizer and runs every entry point on small inputs in
  a child Python process with the sanitizer runtimes preloaded.

A sanitizer finding makes the program exit non-zero with its report.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
import textwrap

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2608_27460_amd", "csrc")
SAN = os.path.join(ROOT, "tests", "sanitize")
HOST_SOURCES = [os.path.join(CSRC, f) for f in ("api.cpp", "builder.cpp", "index_io.cpp")] + \
    [os.path.join(SAN, f) for f in ("device_stubs.cpp", "host_driver.cpp")]
HIP_INCLUDE = "/opt/rocm/include"


def _runtime(name: str) -> str | None:
    p = subprocess.run(["gcc", "-print-file-name=" + name], capture_output=True, text=True).stdout.strip()
    return p if os.path.isabs(p) and os.path.exists(p) else None


def _need_toolchain():
    if not shutil.which("g++") or not shutil.which("gcc"):
        pytest.skip("no host compiler")
    if not os.path.exists(os.path.join(HIP_INCLUDE, "hip", "hip_runtime.h")):
        pytest.skip("HIP headers not found")


def _build_host(tmp_path, flags: list) -> str:
    exe = str(tmp_path / "host_driver")
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer", "-pthread", "-D__HIP_PLATFORM_AMD__",
           "-I", HIP_INCLUDE, "-I", os.path.join(ROOT, "include"), "-I", CSRC] + flags + HOST_SOURCES + ["-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    return exe


def _run(cmd, env=None, timeout=240):
    r = subprocess.run(cmd, capture_output=True, text=True, env=env, timeout=timeout)
    assert r.returncode == 0, "exit %d\n%s\n%s" % (r.returncode, r.stdout[-2000:], r.stderr[-6000:])
    return r.stdout


def test_host_runtime_asan_ubsan(tmp_path):
    _need_toolchain()
    if not _runtime("libasan.so") or not _runtime("libubsan.so"):
        pytest.skip("no ASan/UBSan runtime")
    exe = _build_host(tmp_path, ["-fsanitize=address,undefined", "-fno-sanitize-recover=all"])
    scratch = tmp_path / "files"
    scratch.mkdir()
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")
    assert "all checks passed" in _run([exe, str(scratch)], env)


def test_host_runtime_tsan(tmp_path):
    _need_toolchain()
    if not _runtime("libtsan.so"):
        pytest.skip("no TSan runtime")
    exe = _build_host(tmp_path, ["-fsanitize=thread"])
    scratch = tmp_path / "files"
    scratch.mkdir()
    env = dict(os.environ, TSAN_OPTIONS="halt_on_error=1")
    assert "all checks passed" in _run([exe, str(scratch)], env)


ORACLE_SCRIPT = textwrap.dedent("""
    import os, sys, tempfile
    import numpy as np
    sys.path.insert(0, sys.argv[1])
    import oracle.build as B
    B.LIB = sys.argv[2]
    from oracle import oracle as O
    from paper_2608_27460_amd import synth
    assert O.lib()._name == sys.argv[2], O.lib()._name
    for dt, d in ((synth.F32, 24), (synth.BF16, 32)):
        W = synth.make_w(600, d, dt, 7)
        H, _ = synth.make_queries(W, dt, 5, 8)
        ids, lg, _ = O.topk(W, dt, H, 10)
        O.scores(W, dt, H[:1])
        O.scatter(ids, lg, 600)
        g = O.hnsw_build(W, dt, 8, 40, 3)
        assert O.check_graph(g) == ""
        g1 = O.hnsw_build(W, dt, 6, 30, 3, M0=20, select="simple")
        assert O.check_graph(g1) == ""
        O.hnsw_search(W, dt, g, H, 10, 50, trace_cap=128)
        O.hnsw_search_multi(W, dt, g, H, 10, 50, 8, trace_cap=256)
        qw, qs = O.quantize_rows(W, dt)
        O.hnsw_search_q(W, dt, g, qw, qs, H, 10, 50, expand_width=4)
        O.forced_merge(W, dt, H, ids, np.array([0, 5, 599], np.int32))
        O.knn_graph(W, dt, 12, 16, with_forward=True)
        with tempfile.TemporaryDirectory() as t:
            p = os.path.join(t, "g.vie")
            O.save_graph(g, p, W)
            g2, fp = O.load_graph(p)
            assert fp == O.fingerprint(W, dt)
            assert np.array_equal(g2.adj0, g.adj0)
    print("oracle: all entry points ran")
""")


def test_oracle_asan_ubsan(tmp_path):
    _need_toolchain()
    asan, ubsan = _runtime("libasan.so"), _runtime("libubsan.so")
    if not asan or not ubsan:
        pytest.skip("no ASan/UBSan runtime")
    lib = str(tmp_path / "liboracle_san.so")
    r = subprocess.run(["gcc", "-O1", "-g", "-std=c11", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
                        "-fno-sanitize-recover=all", "-shared", "-fPIC", os.path.join(ROOT, "oracle", "oracle.c"),
                        "-o", lib, "-lm"], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    script = tmp_path / "drive_oracle.py"
    script.write_text(ORACLE_SCRIPT)
    # the interpreter is not instrumented: its own allocations are not checked for leaks
    env = dict(os.environ, LD_PRELOAD=asan + " " + ubsan, ASAN_OPTIONS="detect_leaks=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    assert "all entry points ran" in _run([sys.executable, str(script), ROOT, lib], env)
