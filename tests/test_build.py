"""CPU check of the gfx950 code the build produces: no kernel keeps values in scratch memory.

A kernel that spills registers, or whose compiler turned a small register array into an indexed
stack array, reads and writes per-lane scratch in its loop and loses a large part of its HBM
rate.  hipcc's resource-usage remarks report both per kernel.
"""
import os
import re
import subprocess
from concurrent.futures import ThreadPoolExecutor

import pytest

from paper_2607_21475_amd import build

SOURCES = [s for s in build.SOURCES if s.endswith(".hip")]


def _usage(src):
    cmd = [build.HIPCC, *build.FLAGS, "-c", os.path.join(build.CSRC, src), "-o", os.devnull,
           "-Rpass-analysis=kernel-resource-usage"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    kernels, cur = {}, None
    for line in r.stderr.splitlines():
        m = re.search(r"Function Name: (\S+)", line)
        if m:
            cur = m.group(1)
            kernels[cur] = {}
            continue
        m = re.search(r"remark:\s+(ScratchSize \[bytes/lane\]|VGPRs Spill|SGPRs Spill): (\d+)", line)
        if m and cur:
            kernels[cur][m.group(1)] = int(m.group(2))
    return kernels


@pytest.mark.skipif(not os.path.exists(build.HIPCC), reason="hipcc not installed")
def test_no_kernel_uses_scratch():
    with ThreadPoolExecutor(max_workers=len(SOURCES)) as ex:
        usage = dict(zip(SOURCES, ex.map(_usage, SOURCES)))
    seen = 0
    for src, kernels in usage.items():
        for name, u in kernels.items():
            seen += 1
            assert u.get("ScratchSize [bytes/lane]", 0) == 0, (src, name, u)
            assert u.get("VGPRs Spill", 0) == 0, (src, name, u)
    assert seen >= 10  # the kernels of every source were reported
