"""Host-side robustness of the library's C++ (no GPU).

* The prefix tree on a path with 200,000 branch points, run with a 1 MiB
  stack under the address and undefined-behaviour sanitizers: counting,
  matching, evicting a deep subtree and teardown work level by level without
  recursion (tests/native/prefix_tree_deep.cpp).
* The host code of libhswa (the C ABI's argument validation, the allocator,
  the prefix tree) built with the same sanitizers and run under the CPU tests
  that drive it through the C ABI: test_allocator.py, test_prefix_tree.py and
  test_abi.py must pass with no sanitizer report.
"""

import os
import resource
import subprocess
import sys

import pytest

from paper_2607_13095_amd import build_lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
pytestmark = pytest.mark.skipif(not build_lib.CXX or not os.path.exists(build_lib.CXX), reason="no host C++ compiler")


def _small_stack():
    resource.setrlimit(resource.RLIMIT_STACK, (1 << 20, 1 << 20))


def test_prefix_tree_deep_path(tmp_path):
    exe = str(tmp_path / "prefix_tree_deep")
    build_lib._run([build_lib.CXX, "-std=c++17", *build_lib.SAN_FLAGS, "-Wno-subobject-linkage",
                    "-I", os.path.join(ROOT, "include"), os.path.join(ROOT, "tests", "native", "prefix_tree_deep.cpp"),
                    "-o", exe])
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1")
    r = subprocess.run([exe, "200000"], preexec_fn=_small_stack, capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode == 0 and r.stdout.startswith("ok 200000"), r.stdout + r.stderr[-3000:]


def test_host_code_under_sanitizers(tmp_path):
    lib = build_lib.build_host_sanitized(str(tmp_path))
    files = [os.path.join("tests", f) for f in ("test_allocator.py", "test_prefix_tree.py", "test_abi.py")]
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-m", "not gpu", "-p", "no:cacheprovider", *files],
                       cwd=ROOT, env=build_lib.sanitizer_env(lib), capture_output=True, text=True, timeout=600)
    tail = (r.stdout + r.stderr)[-4000:]
    assert r.returncode == 0, tail
    assert "ERROR: AddressSanitizer" not in r.stderr and "runtime error" not in r.stderr, tail
    # the run loaded the sanitizer build, not libhswa.so
    probe = subprocess.run([sys.executable, "-c", "from paper_2607_13095_amd import hswa; hswa.load();"
                            "print(any('libhswa_san.so' in l for l in open('/proc/self/maps')))"],
                           cwd=ROOT, env=build_lib.sanitizer_env(lib), capture_output=True, text=True, timeout=300)
    assert probe.stdout.strip().endswith("True"), probe.stdout + probe.stderr[-2000:]
