"""The C-ABI from plain C: tests/c_consumer.c is compiled as C99 against
include/hilore.h (warnings are errors), linked against the in-tree
libhilore.so and run.  It only makes calls that return before anything
reaches a device, so it runs without a GPU."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIBDIR = os.path.join(ROOT, "paper_2609_33570_amd")


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
def test_plain_c_consumer(tmp_path):
    assert os.path.exists(os.path.join(LIBDIR, "libhilore.so")), "build() first"
    exe = tmp_path / "c_consumer"
    subprocess.run(["gcc", "-std=c99", "-Wall", "-Wextra", "-pedantic", "-Werror",
                    "-I", os.path.join(ROOT, "include"), os.path.join(ROOT, "tests", "c_consumer.c"),
                    "-L", LIBDIR, "-lhilore", f"-Wl,-rpath,{LIBDIR}", "-o", str(exe)], check=True)
    res = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120)
    assert res.returncode == 0, res.stdout + res.stderr
    assert res.stdout.strip().endswith("OK")
