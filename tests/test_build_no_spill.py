"""The hot kernels keep every value in registers: no kernel of libzo spills to scratch memory.

Compiles each HIP source's device code for gfx950 to assembly (the flags of the library build)
and reads the private segment size the compiler assigns each kernel.  A spill there once hid a
miscompiled accumulator copy in an epilogue, and spills cost memory traffic in the loops, so any
nonzero size fails."""
import glob
import os
import re
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
from paper_2608_15665_amd import _build  # noqa: E402


def _asm(src, tmp):
    out = os.path.join(tmp, os.path.basename(src) + ".s")
    flags = [f for f in _build.HIPCC_FLAGS if f != "-fPIC"]
    cmd = [_build.hipcc(), *flags, *_build.FILE_FLAGS.get(os.path.basename(src), []), "--cuda-device-only", "-S",
           src, "-o", out]
    p = subprocess.run(cmd, capture_output=True, text=True)
    assert p.returncode == 0, p.stderr[-2000:]
    return open(out).read()


def test_no_kernel_spills(tmp_path):
    try:
        _build.hipcc()
    except RuntimeError:
        pytest.skip("hipcc not available")
    srcs = sorted(glob.glob(os.path.join(_build.CSRC, "*.hip")))
    with ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        texts = list(ex.map(lambda s: _asm(s, str(tmp_path)), srcs))
    kernels, spills = 0, []
    for src, text in zip(srcs, texts):
        for m in re.finditer(r"\.amdhsa_kernel (\S+)(.*?)\.end_amdhsa_kernel", text, re.S):
            kernels += 1
            size = int(re.search(r"\.amdhsa_private_segment_fixed_size (\d+)", m.group(2)).group(1))
            if size:
                spills.append((os.path.basename(src), m.group(1), size))
    assert kernels > 20
    assert not spills, spills
