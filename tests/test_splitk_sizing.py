"""Split-K workspace sizing against the dispatch heuristic (CPU only): builds
tests/native/splitk_sizing.cpp, which includes the library's loss and block
sources and calls their own workspace carving, and runs it on the host
(nothing is launched).  Regression: the LM head's weight-gradient product
once split its last, narrower vocab chunk into a workspace carved for the
full chunks only."""
import os
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
LIBDIR = os.path.join(ROOT, "paper_2606_04484_amd")


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not installed")
@pytest.mark.skipif(not os.path.exists(os.path.join(LIBDIR, "libaj.so")), reason="libaj.so not built")
def test_splitk_partials_fit_workspace(tmp_path):
    exe = str(tmp_path / "splitk_sizing")
    src = os.path.join(ROOT, "tests", "native", "splitk_sizing.cpp")
    r = subprocess.run([HIPCC, "-O1", "-std=c++17", "--offload-arch=gfx950", "-Xclang",
                        "-target-feature", "-Xclang", "-packed-fp32-ops",
                        "-I", os.path.join(ROOT, "include"), "-I", os.path.join(LIBDIR, "csrc"),
                        "-x", "hip", src, "-o", exe, "-L", LIBDIR, "-laj",
                        "-Wl,-rpath," + LIBDIR], capture_output=True, text=True, cwd=str(tmp_path))
    assert r.returncode == 0, r.stderr[-2000:]
    r = subprocess.run([exe], capture_output=True, text=True, timeout=300)
    print(r.stdout)
    assert r.returncode == 0 and "violations: 0" in r.stdout
