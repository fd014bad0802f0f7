"""The host-side data preparation (weight packing into matrix-fragment order,
workspace layouts, segment-table checks; paper_2606_09312_amd/csrc/
wm_pack.cpp) built on its own with the address and undefined-behaviour
sanitizers and driven by tests/host/pack_check.cpp over every instantiated
shape and both transition forms: packed chunks against direct matrix
products through the matrix-core operand conventions, narrow and transposed
blobs as exact permutations of their matrices, workspace parts aligned and
disjoint, segment tables accepted and rejected as documented."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2606_09312_amd", "csrc")


@pytest.mark.skipif(shutil.which("g++") is None, reason="g++ not available")
def test_pack_and_layouts_under_sanitizers(tmp_path):
    exe = str(tmp_path / "pack_check")
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all", f"-I{CSRC}",
           os.path.join(ROOT, "tests", "host", "pack_check.cpp"), os.path.join(CSRC, "wm_pack.cpp"),
           "-o", exe]
    res = subprocess.run(cmd, capture_output=True, text=True)
    assert res.returncode == 0, res.stderr[-4000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    run = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=600)
    print(run.stdout[-2000:])
    assert run.returncode == 0, (run.stdout[-2000:], run.stderr[-4000:])
    assert "all ok" in run.stdout
