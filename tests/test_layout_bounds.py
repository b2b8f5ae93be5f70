"""The host layout under a bounds-checked CPU build.

tests/layout_bounds_main.cpp links the library's layout code (csrc/layout.cpp) into a host
program built with the address and undefined-behaviour sanitizers (recovery off) and the
C++ library's container assertions, builds the layout of seeded inputs under many
parameter sets (units, LDS cells, hot-item cells, dense tiles, the sequential order,
minibatch blocks, worker classes, padded ranks 8 to 512, a one-rating matrix and an empty
one) and runs the layout's self-check on every block.  No GPU is involved.
"""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs the host C++ compiler")
def test_layout_under_address_and_ub_sanitizers(tmp_path):
    exe = str(tmp_path / "layout_bounds")
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-pthread", "-fno-omit-frame-pointer", "-D_GLIBCXX_ASSERTIONS",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           os.path.join(HERE, "layout_bounds_main.cpp"), os.path.join(ROOT, "paper_1410_8043_amd", "csrc", "layout.cpp"),
           "-o", exe]
    subprocess.run(cmd, check=True)
    # the environment is passed on as it is; the sanitizer runtime is told not to insist on
    # coming first among the preloaded libraries
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:verify_asan_link_order=0", UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=600)
    assert r.returncode == 0, (r.stdout[-4000:], r.stderr[-4000:])
    assert "0 failures" in r.stdout
