"""Host-side check of the weight-gradient kernel's generated code.

The DMA-staged weight-gradient kernel issues its transposing LDS reads
(``ds_read_b64_tr_b16``) from inline assembly, so the compiler does not know
that their destination registers fill in asynchronously: only the kernel's
own ``s_waitcnt lgkmcnt(N)`` makes them valid.  If the compiler ever placed
an instruction that touches such a register (an MFMA, a register copy, a
reuse) between the read and a wait that covers it, the kernel would read
stale data without any error.  This test compiles the source with the
library's flags and walks every path of the generated code from each such
read: the first instruction that names a destination register must come
after an ``s_waitcnt`` whose lgkmcnt is at most the number of LDS
instructions issued after the read on that path (LDS operations of one wave
complete in order, so that wait covers it).
"""

from __future__ import annotations

import os
import re
import shutil
import subprocess

import pytest

from paper_1911_07384_amd import build as B

VREG = re.compile(r"\bv\[(\d+):(\d+)\]|\bv(\d+)\b")
LGKM = re.compile(r"lgkmcnt\((\d+)\)")


def _kernels(asm: str) -> dict[str, list[str]]:
    """Instruction and label lines of each kernel, comments stripped."""
    out: dict[str, list[str]] = {}
    cur = None
    for raw in asm.splitlines():
        line = raw.split(";", 1)[0].rstrip()
        if not line.strip():
            continue
        if not line.startswith((" ", "\t")) and line.endswith(":") and not line.startswith("."):
            cur = line[:-1]
            out[cur] = []
            continue
        if cur is None:
            continue
        s = line.strip()
        if s.startswith(".LBB") and s.endswith(":"):
            out[cur].append(s)
        elif not s.startswith("."):
            out[cur].append(s)
            if s.startswith("s_endpgm"):
                cur = None
    return out


def _regs(operands: str) -> set[int]:
    r: set[int] = set()
    for m in VREG.finditer(operands):
        if m.group(3) is not None:
            r.add(int(m.group(3)))
        else:
            r.update(range(int(m.group(1)), int(m.group(2)) + 1))
    return r


def _check_kernel(lines: list[str]) -> int:
    """Number of transposing reads verified; raises on a violation."""
    labels = {l[:-1]: i for i, l in enumerate(lines) if l.endswith(":")}
    checked = 0
    for i, l in enumerate(lines):
        if not l.startswith("ds_read_b64_tr_b16"):
            continue
        dst = _regs(l.split(None, 1)[1].split(",")[0])
        stack = [(i + 1, 0)]
        seen = set()
        while stack:
            pos, after = stack.pop()
            while pos < len(lines):
                if (pos, after) in seen:
                    break
                seen.add((pos, after))
                ins = lines[pos]
                if ins.endswith(":"):
                    pos += 1
                    continue
                op, _, args = ins.partition(" ")
                if op == "s_waitcnt":
                    m = LGKM.search(args)
                    if (m and int(m.group(1)) <= after) or args.strip() == "0":
                        break  # covered on this path
                if _regs(args) & dst:
                    raise AssertionError(
                        f"{ins!r} (line {pos}) uses a register of {l!r} (line {i}) "
                        "before a wait covers it")
                if op.startswith("ds_"):
                    after += 1
                if op == "s_endpgm":
                    break
                if op == "s_branch":
                    pos = labels[args.strip()]
                    continue
                if op.startswith("s_cbranch"):
                    stack.append((labels[args.strip()], after))
                pos += 1
        checked += 1
    return checked


@pytest.mark.skipif(not os.path.exists(B.HIPCC) and shutil.which("hipcc") is None,
                    reason="hipcc not available")
def test_wgrad_transposing_reads_are_waited_for(tmp_path):
    out = tmp_path / "conv_wgrad.s"
    flags = [f for f in B.FLAGS if f != "-fPIC"]
    cmd = [B.HIPCC, *flags, "--cuda-device-only", "-S",
           os.path.join(B.CSRC, "conv_wgrad.hip"), "-o", str(out)]
    subprocess.run(cmd, check=True, capture_output=True)
    kernels = _kernels(out.read_text())
    wg7 = {k: v for k, v in kernels.items() if "wgrad7_kernel" in k}
    assert len(wg7) >= 8, sorted(kernels)
    for name, lines in wg7.items():
        n = _check_kernel(lines)
        assert n >= 8, (name, n)


def test_checker_flags_an_early_use():
    # a read whose register is copied before the covering wait must fail,
    # one read behind a sufficient wait must pass, and a wait that still lets
    # the read be in flight does not count
    bad = ["ds_read_b64_tr_b16 v[6:7], v2 offset:512", "v_mov_b32 v40, v6",
           "s_waitcnt lgkmcnt(0)", "s_endpgm"]
    with pytest.raises(AssertionError):
        _check_kernel(bad)
    good = ["ds_read_b64_tr_b16 v[6:7], v2", "ds_read_b64_tr_b16 v[8:9], v2 offset:512",
            "s_waitcnt lgkmcnt(1)", "v_mov_b32 v40, v6", "s_waitcnt lgkmcnt(0)",
            "v_mov_b32 v41, v8", "s_endpgm"]
    assert _check_kernel(good) == 2
    loose = ["ds_read_b64_tr_b16 v[6:7], v2", "ds_read_b64_tr_b16 v[8:9], v2 offset:512",
             "s_waitcnt lgkmcnt(2)", "v_mov_b32 v40, v6", "s_endpgm"]
    with pytest.raises(AssertionError):
        _check_kernel(loose)
    # a use reached only through a branch back to a label is found too
    loop = [".LBB0_1:", "v_mov_b32 v40, v6", "ds_read_b64_tr_b16 v[6:7], v2",
            "s_cbranch_scc1 .LBB0_1", "s_waitcnt lgkmcnt(0)", "s_endpgm"]
    with pytest.raises(AssertionError):
        _check_kernel(loop)
