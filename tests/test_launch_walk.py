"""Host build of the apply launch decomposition (tests/host_checks/launch_walk.cpp,
g++ with AddressSanitizer and UBSan): the tiles cover each batch, and every
shrink / expand work item of a launch is enumerated exactly once over ranges
that partition each table."""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(os.path.dirname(HERE), "paper_2608_03579_amd", "csrc")


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_launch_walk(tmp_path):
    exe = str(tmp_path / "launch_walk")
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-DSALT_HOST_ONLY", "-fsanitize=address,undefined",
           "-fno-sanitize-recover=undefined", f"-I{CSRC}", os.path.join(HERE, "host_checks", "launch_walk.cpp"),
           "-o", exe]
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    res = subprocess.run([exe], capture_output=True, text=True, timeout=600)
    assert res.returncode == 0 and res.stdout.strip().endswith("ok"), res.stdout + res.stderr
