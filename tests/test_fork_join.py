"""Host test of the library's two-stream ordering (csrc/fork_join.hpp):
compiled with g++ against stand-in stream operations that record every call
and inject failures; checks that once work is on the side stream the
caller's stream always waits for it, on the error paths too."""
import os
import shutil
import subprocess
import tempfile

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(ROOT, "paper_2607_20214_amd", "csrc")
ROCM_INC = "/opt/rocm/include"


@pytest.mark.skipif(shutil.which("g++") is None or not os.path.isdir(ROCM_INC), reason="needs g++ and the HIP headers")
def test_fork_join_orders_main_after_side_on_every_path():
    with tempfile.TemporaryDirectory() as d:
        exe = os.path.join(d, "fork_join_check")
        subprocess.run(["g++", "-std=c++17", "-O1", "-Wall", "-D__HIP_PLATFORM_AMD__", "-I", ROCM_INC, "-I", CSRC,
                        os.path.join(HERE, "host", "fork_join_check.cpp"), "-o", exe], check=True)
        r = subprocess.run([exe], capture_output=True, text=True)
        print(r.stdout)
        assert r.returncode == 0, r.stdout + r.stderr
        assert "ALL OK" in r.stdout
