"""Compile-time checks of the gfx950 kernels (CPU only): no kernel keeps
private arrays in scratch memory or spills registers -- register stages that
fall back to scratch turn every streamed byte into extra memory traffic."""
import glob
import os
import re
import subprocess

import pytest

from paper_2609_32395_amd import build as B


def _resource_remarks(src):
    cmd = [B.HIPCC, *B.COMMON_FLAGS, "-c", src, "-o", os.devnull, "-Rpass-analysis=kernel-resource-usage"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    kernels = {}
    name = None
    for line in r.stderr.splitlines():
        m = re.search(r"Function Name: (\S+)", line)
        if m:
            name = m.group(1)
            kernels[name] = {}
            continue
        m = re.search(r"remark:\s+(.+?): (\d+)", line)
        if m and name:
            kernels[name][m.group(1).strip()] = int(m.group(2))
    return kernels


@pytest.mark.parametrize("src", sorted(glob.glob(os.path.join(B.CSRC, "*.hip"))), ids=os.path.basename)
def test_no_scratch_no_spills(src):
    ks = _resource_remarks(src)
    for name, res in ks.items():
        assert res.get("ScratchSize [bytes/lane]", 0) == 0, (name, res)
        assert res.get("VGPRs Spill", 0) == 0 and res.get("SGPRs Spill", 0) == 0, (name, res)
