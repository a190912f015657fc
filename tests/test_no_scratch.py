"""Every kernel of the library runs without scratch (private) memory: a register spill or
an array indexed at run time would put its loads and stores behind the same memory counter
as the direct-to-LDS loads, whose waits the kernels place by hand, and costs a memory round
trip per use.  Each HIP source is compiled for gfx950 (device code only) with the compiler's
resource report, and every kernel's scratch size must be 0.  (CPU only.)"""
import concurrent.futures as cf
import os
import re
import shutil
import subprocess

import pytest

from paper_2605_30218_amd import build_lib

pytestmark = pytest.mark.skipif(shutil.which("hipcc") is None, reason="hipcc not on PATH")


def _report(src):
    cmd = ["hipcc", *build_lib.FLAGS, "--cuda-device-only", "-c", src, "-o", os.devnull,
           "-Rpass-analysis=kernel-resource-usage"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    kernels, name = {}, None
    for line in r.stderr.splitlines():
        m = re.search(r"Function Name: (\S+)", line)
        if m:
            name = m.group(1)
        m = re.search(r"ScratchSize \[bytes/lane\]: (\d+)", line)
        if m and name:
            kernels[name] = int(m.group(1))
    return src, kernels


def test_no_kernel_uses_scratch_memory():
    srcs = build_lib.sources()
    with cf.ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        reports = list(ex.map(_report, srcs))
    n = sum(len(k) for _, k in reports)
    assert n > 50, "the resource report names the kernels"
    bad = {f"{os.path.basename(s)}:{k}": v for s, ks in reports for k, v in ks.items() if v}
    assert not bad, f"kernels with scratch memory: {bad}"
