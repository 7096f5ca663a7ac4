"""No kernel of the library uses private (scratch) memory.

A kernel whose argument struct or locals spill to scratch still computes the
right bytes, so the parity tests cannot see it, but every lane then streams
its copy through memory: a gather whose 1.4 KB argument block was copied to
scratch ran 20 times slower.  The compiler's resource-usage remarks for the
gfx950 build of every library source must report a scratch size of 0 for
every kernel (CPU only: hipcc cross-compiles)."""
import os
import re
import subprocess

import pytest

from paper_2310_05205_amd import build

REMARK = re.compile(r"remark:\s+(Function Name: (\S+)|ScratchSize \[bytes/lane\]: (\d+))")


def _resource_remarks(source):
    hipcc = os.environ.get("HIPCC", "hipcc")
    cmd = [hipcc, "--offload-arch=gfx950", "-O3", "-std=c++17", "--cuda-device-only", "-c", "-o", os.devnull,
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-I" + build.INCLUDE, "-I" + build.CSRC, "-Rpass-analysis=kernel-resource-usage",
           os.path.join(build.CSRC, source)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    scratch, name = {}, None
    for m in REMARK.finditer(r.stderr):
        if m.group(2):
            name = m.group(2)
        elif name is not None:
            scratch[name] = int(m.group(3))
    return scratch


@pytest.mark.parametrize("source", build.SOURCES)
def test_no_kernel_uses_scratch(source):
    scratch = _resource_remarks(source)
    if source != "table.hip":  # host-only code, no kernels
        assert scratch, "no kernel resource remarks for %s" % source
    assert {k: v for k, v in scratch.items() if v} == {}
