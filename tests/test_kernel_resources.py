"""Register and scratch budgets of the HIP kernels (no GPU: compiles for gfx950).

The MFMA kernels are written for a fixed occupancy (two waves per SIMD for the
convolution and weight-gradient kernels) and keep their accumulators in
registers; a change that makes the compiler spill registers or place an array in
scratch memory still computes the right values but loses a large part of the
speed.  These tests compile each source with the compiler's resource report
and check every kernel: no scratch, no spilled vector registers, and at least
two waves per SIMD for the MFMA kernels."""
import concurrent.futures as cf
import os
import re
import shutil
import subprocess

import pytest

from paper_1508_06904_amd import build

SOURCES = ["conv_mfma.hip", "backward.hip", "conv_direct.hip", "kernels_data.hip"]


def _report(src):
    cmd = [build.HIPCC, "-x", "hip"] + build.FLAGS + ["-c", os.path.join(build.CSRC, src), "-o", os.devnull,
                                                      "-Rpass-analysis=kernel-resource-usage"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    kernels, cur = {}, None
    for line in r.stderr.splitlines():
        m = re.search(r"remark: Function Name: (\S+)", line)
        if m:
            cur = m.group(1)
            kernels[cur] = {}
            continue
        m = re.search(r"remark:\s+([A-Za-z ]+?)(?: \[[^\]]*\])?: (\d+)", line)
        if cur and m:
            kernels[cur][m.group(1).strip()] = int(m.group(2))
    return kernels


@pytest.fixture(scope="module")
def reports():
    if not os.path.exists(build.HIPCC) and shutil.which(build.HIPCC) is None:
        pytest.skip("hipcc not available")
    with cf.ThreadPoolExecutor(max_workers=len(SOURCES)) as ex:
        return dict(zip(SOURCES, ex.map(_report, SOURCES)))


@pytest.mark.parametrize("src", SOURCES)
def test_no_scratch_and_no_spills(reports, src):
    ks = reports[src]
    assert ks, "no kernels reported for %s" % src
    for name, r in ks.items():
        assert r.get("ScratchSize", 0) == 0, (name, r)
        # (scalar registers spill into vector-register lanes, not to memory)
        assert r.get("VGPRs Spill", 0) == 0, (name, r)


def test_mfma_kernels_keep_two_waves_per_simd(reports):
    mfma = {n: r for src in ("conv_mfma.hip", "backward.hip") for n, r in reports[src].items()
            if "conv_mfma_kernel" in n or "wgrad_mfma_kernel" in n}
    assert len(mfma) >= 20
    for name, r in mfma.items():
        assert r["Occupancy"] >= 2, (name, r)
