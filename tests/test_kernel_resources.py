"""Every kernel of the library runs without scratch (private) memory.

Scratch on gfx950 is per-lane memory behind the vector memory path: a kernel that spills registers or keeps a
local array or struct it indexes by a lane-varying value there pays hundreds of cycles per access.  The
compiler's resource remarks (-Rpass-analysis=kernel-resource-usage) report each kernel's scratch size; this
compiles every source for gfx950 (device code only, as the build does) and checks them all.  Host-only: no GPU."""
import concurrent.futures as cf
import glob
import os
import re
import shutil
import subprocess
import tempfile

import pytest

from paper_1702_02181_amd import build_lib as B


def _remarks(src, out_dir):
    obj = os.path.join(out_dir, os.path.basename(src) + ".o")
    r = subprocess.run([B.HIPCC, *B.COMMON, "--cuda-device-only", "-c", "-Rpass-analysis=kernel-resource-usage",
                        src, "-o", obj], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    return r.stderr


@pytest.mark.skipif(shutil.which(B.HIPCC) is None and not os.path.exists(B.HIPCC), reason="hipcc not available")
def test_no_kernel_uses_scratch():
    srcs = sorted(glob.glob(os.path.join(B.CSRC, "*.hip")))
    assert srcs
    with tempfile.TemporaryDirectory() as d, cf.ThreadPoolExecutor(min(8, len(srcs))) as ex:
        outs = list(ex.map(lambda s: _remarks(s, d), srcs))
    kernels, scratch = 0, {}
    for text in outs:
        name = None
        for line in text.splitlines():
            m = re.search(r"Function Name: (\S+)", line)
            if m:
                name = m.group(1)
                continue
            m = re.search(r"ScratchSize \[bytes/lane\]: (\d+)", line)
            if m and name:
                kernels += 1
                if int(m.group(1)):
                    scratch[name] = int(m.group(1))
    assert kernels > 50, "no resource remarks parsed"
    assert not scratch, f"kernels using scratch memory: {scratch}"
