"""Build-time resource check of the HIP kernels (CPU only: hipcc cross-compiles).

No kernel may use scratch (private segment) memory: a launch of a kernel that
does must first set up scratch for every wave, which makes every apply slower.
Scratch appears when registers spill or when a struct whose address escapes is
copied out of the kernel arguments.
"""
import os
import re
import shutil
import subprocess
import tempfile

import pytest

from paper_2608_03579_amd import build

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.skipif(not os.path.exists(build.hipcc()), reason="hipcc not installed")
def test_no_kernel_uses_scratch():
    meta = ""
    with tempfile.TemporaryDirectory() as d:
        for src in build.SOURCES:
            if not src.endswith(".hip"):
                continue
            out = os.path.join(d, os.path.basename(src) + ".s")
            flags = [f for f in build.HIPCC_FLAGS if f not in ("-shared", "-fPIC")]
            cmd = [build.hipcc(), *flags, "--cuda-device-only", "-S", src, "-o", out]
            res = subprocess.run(cmd, capture_output=True, text=True)
            assert res.returncode == 0, res.stderr[-2000:]
            meta += open(out).read()
    kernels = re.findall(r"\.name:\s+(\S+)\n(.*?)(?=\n  - \.|\Z)", meta, re.S)
    kernels = [(n, b) for n, b in kernels if any(k in n for k in ("k_shrink", "k_expand", "k_plan", "k_fuse",
                                                                   "k_gram"))]
    assert len(kernels) >= 100, f"only {len(kernels)} kernels found"
    for name, body in kernels:
        priv = int(re.search(r"\.private_segment_fixed_size:\s+(\d+)", body).group(1))
        spills = int(re.search(r"\.vgpr_spill_count:\s+(\d+)", body).group(1))
        assert priv == 0 and spills == 0, f"{name}: {priv} bytes of scratch, {spills} VGPR spills"
