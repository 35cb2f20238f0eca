"""The decode kernels' untracked page-id loads (no GPU; hipcc only).

The 128-row decode kernel fetches each step's page id with a scalar load
issued as inline assembly at the end of a step and waited for (s_waitcnt
lgkmcnt(0)) inside the next step's barrier, so that the load's latency
overlaps the end of the step.  The compiler does not know that the load is
still in flight after the statement that issues it: it could read the
destination register, copy it, or reuse it for another value before the
wait.  This test builds decode_attn.hip to gfx950 assembly with the
library's flags and walks every path from each such load to its wait in
every decode kernel: no instruction on the way may name the register.
"""
import os
import re
import shutil
import subprocess

import pytest

from paper_2609_36760_amd import build as b

HIPCC = os.path.join(b.ROCM, "bin", "hipcc")

pytestmark = pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not installed")


def _names(reg: int, text: str) -> bool:
    """Whether an instruction's operands name SGPR `reg` (alone or in a range)."""
    for m in re.finditer(r"\bs(\d+)\b|\bs\[(\d+):(\d+)\]", text):
        if m.group(1) is not None and int(m.group(1)) == reg:
            return True
        if m.group(2) is not None and int(m.group(2)) <= reg <= int(m.group(3)):
            return True
    return False


def _walk(lines, labels, start, reg):
    """Instructions on any path from line `start` to a full lgkmcnt wait that name `reg`."""
    bad, seen, todo = [], set(), [start + 1]
    while todo:
        i = todo.pop()
        while i < len(lines) and i not in seen:
            seen.add(i)
            ins = lines[i].split(";")[0].strip()
            if not ins or ins.endswith(":") or ins.startswith("."):
                i += 1
                continue
            op = ins.split()[0]
            if op == "s_waitcnt" and "lgkmcnt(0)" in ins:
                break
            if _names(reg, ins.partition(" ")[2]):
                bad.append((i, ins))
            if op == "s_endpgm":
                break
            if op == "s_branch":
                i = labels[ins.split()[1]]
                continue
            if op.startswith("s_cbranch"):
                todo.append(labels[ins.split()[1]])
            i += 1
    return bad


def test_page_id_register_untouched_until_its_wait(tmp_path):
    src = os.path.join(b.CSRC, "decode_attn.hip")
    out = tmp_path / "decode_attn.s"
    r = subprocess.run([HIPCC, *b.HIP_FLAGS, "--cuda-device-only", "-S", src, "-o", str(out)],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    asm = out.read_text()
    kernels = re.findall(r"^(_ZN\w*decode_kernel\w*):", asm, flags=re.M)
    assert len(kernels) >= 9, kernels
    checked = 0
    for name in kernels:
        body = asm[asm.index(name + ":"):]
        body = body[:body.index(".Lfunc_end")]
        lines = body.split("\n")
        labels = {l.split(":")[0]: i for i, l in enumerate(lines) if re.match(r"^\.LBB\w+:", l)}
        for i, l in enumerate(lines):
            # the inline page-id loads: an SGPR offset (the compiler's own loads use immediates)
            m = re.match(r"\s*s_load_dword s(\d+), s\[\d+:\d+\], s\d+\s*$", l.split(";")[0])
            if m:
                bad = _walk(lines, labels, i, int(m.group(1)))
                assert not bad, f"{name}: page id in s{m.group(1)} (line {i}) named before its wait: {bad[:3]}"
                checked += 1
    assert checked >= 9 * 4, checked
    # the walk sees a use placed on the way to the wait, also behind a branch
    lines = ["\ts_load_dword s54, s[6:7], s10", "\ts_cbranch_scc1 .LBB0_2", "\ts_branch .LBB0_1",
             ".LBB0_2:", "\ts_add_u32 s3, s[54:55], 4", ".LBB0_1:", "\ts_waitcnt vmcnt(3) lgkmcnt(0)", "\ts_endpgm"]
    labels = {".LBB0_2": 3, ".LBB0_1": 5}
    assert [i for i, _ in _walk(lines, labels, 0, 54)] == [4]
    assert _walk(lines, labels, 0, 53) == []
