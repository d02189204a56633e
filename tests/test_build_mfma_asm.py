"""The GEMM kernels' accumulators stay in place and their inline-asm MFMAs keep their wait states.

k_gemm_main (the fused GEMM) and k_proj (the prepare's projection) issue their MFMAs as inline
assembly with the accumulator tied to the destination (the builtin's untied form made the
register allocator rotate the accumulators through fresh AGPRs and copy them back on every trip
round the loop).  The hazard recognizer does not see
inside inline assembly, so the kernel orders the accumulators through its own fences: zeros
written, then `s_nop 1` (2 wait states) before the first MFMA; after the last MFMA, three
`s_nop 7` (24 wait states) before anything else touches them.  This reads the gfx950 assembly
of every instantiation and checks exactly that layout: every MFMA in place, no other
instruction touching an AGPR between the fences, and the fences in order."""
import os
import re
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
from paper_2608_15665_amd import _build  # noqa: E402

AGPR = re.compile(r"\ba\d+\b|\ba\[\d+:\d+\]")


def _asm(src, tmp):
    out = os.path.join(tmp, os.path.basename(src) + ".s")
    flags = [f for f in _build.HIPCC_FLAGS if f != "-fPIC"]
    cmd = [_build.hipcc(), *flags, *_build.FILE_FLAGS.get(os.path.basename(src), []), "--cuda-device-only", "-S",
           src, "-o", out]
    p = subprocess.run(cmd, capture_output=True, text=True)
    assert p.returncode == 0, p.stderr[-2000:]
    return open(out).read()


def _functions(text, pattern):
    """Instruction lines (comments, labels and directives dropped) of each function matching pattern."""
    funcs, cur = {}, None
    for ln in text.split("\n"):
        m = re.match(r"\s*\.type\s+(\S+),@function", ln)
        if m and re.search(pattern, m.group(1)):
            cur = m.group(1)
            funcs[cur] = []
            continue
        if cur and re.match(r"\s*\.size\s+" + re.escape(cur), ln):
            cur = None
            continue
        t = ln.strip()
        if cur is None or not t or t.startswith((";", ".")) or t.endswith(":"):
            continue
        funcs[cur].append(t)
    return funcs


@pytest.mark.parametrize("kernel,min_kernels,min_mfma", [("k_gemm_main", 12, 256), ("k_proj", 4, 64)])
def test_mfma_in_place_and_fenced(tmp_path, kernel, min_kernels, min_mfma):
    try:
        _build.hipcc()
    except RuntimeError:
        pytest.skip("hipcc not available")
    text = _asm(os.path.join(_build.CSRC, "zo_gemm.hip"), str(tmp_path))
    funcs = _functions(text, kernel + r"I")
    assert len(funcs) >= min_kernels
    for name, ins in funcs.items():
        mfma = [i for i, t in enumerate(ins) if t.startswith("v_mfma")]
        assert len(mfma) >= min_mfma, name
        for i in mfma:
            ops = [o.strip() for o in ins[i].split(None, 1)[1].split(",")]
            assert ops[0] == ops[3], (name, ins[i])  # destination == accumulator source
        init = [i for i, t in enumerate(ins) if t == "s_nop 1"]
        tail = [i for i, t in enumerate(ins) if t == "s_nop 7"]
        assert len(init) >= 8 and len(tail) == 3 and tail[2] - tail[0] == 2, name
        first, last = init[7], tail[0]
        assert first < mfma[0] and mfma[-1] < last, name
        for i in range(first, last):
            t = ins[i]
            if t.startswith(("v_mfma", "s_")):
                continue
            assert not AGPR.search(t), (name, i, t)
        for i in range(0, init[0]):
            assert not ins[i].startswith("v_mfma"), name
        # The zeros are written before the first fence.
        writes = [i for i, t in enumerate(ins) if t.startswith(("v_accvgpr_write", "v_accvgpr_mov"))]
        assert writes and max(writes) < init[0], name
