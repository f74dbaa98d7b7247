"""Generated-code checks of the kernels whose copies are counted by hand (CPU only).

The Softmax -> P.V and attention kernels issue their global->LDS copies from inline
assembly and wait for them with hand-counted `s_waitcnt vmcnt(N)`.  The compiler's
own wait tracking does not see those copies; a wait it places inside a key loop (for
some plain load it believes still pending) also waits, in hardware, for every copy in
flight, which silently turns the copy ring into a synchronous pipeline.  These tests
compile the sources for gfx950 and check that the innermost loops doing matrix work
carry no wait on the vector-memory counter except those written in the source.
"""
import os
import re
import subprocess
import tempfile

import pytest

from paper_2502_17728_amd import build as B


def _have_hipcc():
    try:
        B.hipcc()
        return True
    except RuntimeError:
        return False


pytestmark = pytest.mark.skipif(not _have_hipcc(), reason="hipcc is needed to compile the kernels")


def _device_asm(src):
    with tempfile.TemporaryDirectory() as d:
        out = os.path.join(d, "k.s")
        cmd = [B.hipcc()] + B.common_flags() + ["-S", "--offload-device-only", os.path.join(B.CSRC, src), "-o", out]
        res = subprocess.run(cmd, capture_output=True, text=True)
        assert res.returncode == 0, res.stderr[-2000:]
        return open(out).read()


def _functions(asm, prefix):
    for name in re.findall(r"^(" + prefix + r"\w*):", asm, re.M):
        start = asm.index(name + ":")
        end = asm.index(".Lfunc_end", start)
        yield name, asm[start:end].split("\n")


def _innermost_mfma_loops(body):
    labels = {}
    for i, line in enumerate(body):
        m = re.match(r"^(\.LBB\d+_\d+):", line)
        if m:
            labels[m.group(1)] = i
    loops = set()
    for i, line in enumerate(body):
        m = re.search(r"s_c?branch\w*\s+(\.LBB\d+_\d+)", line)
        if m and m.group(1) in labels and labels[m.group(1)] < i:
            loops.add((labels[m.group(1)], i))
    mfma = [(a, b) for a, b in loops if any("v_mfma" in body[k] for k in range(a, b))]
    # the innermost of those: no other loop with matrix instructions nested inside
    return [(a, b) for a, b in mfma if not any(a <= c and d <= b and (c, d) != (a, b) for c, d in mfma)]


def _compiler_vmcnt_waits(body, a, b):
    """Lines a..b that wait on vmcnt outside inline-assembly blocks."""
    inside = False
    out = []
    for i, line in enumerate(body[: b + 1]):
        if "ASMSTART" in line:
            inside = True
        elif "ASMEND" in line:
            inside = False
        elif i >= a and not inside and re.search(r"s_waitcnt\b.*vmcnt\(", line):
            out.append(line.strip())
    return out


@pytest.mark.parametrize("src,prefix", [("attention.hip", "_ZN2dn16attention_kernel"),
                                        ("softmax_pv.hip", "_ZN2dn17softmax_pv_kernel")])
def test_key_loops_carry_only_hand_counted_waits(src, prefix):
    asm = _device_asm(src)
    seen = 0
    for name, body in _functions(asm, prefix):
        loops = _innermost_mfma_loops(body)
        assert loops, f"{name}: no loop with matrix instructions found"
        for a, b in loops:
            seen += 1
            waits = _compiler_vmcnt_waits(body, a, b)
            assert not waits, f"{name}: compiler-placed vmcnt waits inside a key loop: {waits}"
    assert seen > 0
