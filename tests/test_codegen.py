"""Generated-code check for the matrix-core kernels (CPU only; hipcc cross-compiles).

A VALU instruction that reads an MFMA's destination registers needs several
wait states after the MFMA is issued; the compiler inserts them as s_nop.  A
read that came a single instruction after its MFMA, with a branch in between,
once returned stale values in one lane group (a nearest-distance kernel read
0 where the distance was 493).  This test compiles the MFMA sources with the
library's flags to gfx950 assembly and walks, from every MFMA, the
fall-through path until the first VALU read of its result, counting
instruction slots (s_nop N counts N + 1).  Every such read must be at least
MIN_SLOTS slots after the MFMA; the compiler's own choice on straight-line
code is 8 (bf16 16x16x32) to 10 (fp32 16x16x4).
"""
import concurrent.futures as cf
import os
import re
import subprocess

import pytest

from paper_2004_11127_amd import build

MIN_SLOTS = 6
SOURCES = ["k_small_mfma.hip", "k_mfma.hip", "k_mfma64.hip", "k_knn.hip", "k_small.hip"]


def _asm(src, tmp_path):
    out = os.path.join(tmp_path, src + ".s")
    cmd = [build.HIPCC] + build.flags_for(src) + ["--cuda-device-only", "-S",
                                         os.path.join(build.CSRC, src), "-o", out]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    with open(out) as f:
        return f.read().split("\n")


def _regs(text):
    regs = set()
    for a, b in re.findall(r"v\[(\d+):(\d+)\]", text):
        regs |= set(range(int(a), int(b) + 1))
    for a in re.findall(r"\bv(\d+)\b", text):
        regs.add(int(a))
    return regs


def short_reads(lines):
    """(function, line, slots, instruction) for MFMA results read too soon."""
    found = []
    fn = None
    for i, line in enumerate(lines):
        m = re.match(r"^(_Z\S+):", line)
        if m:
            fn = m.group(1)
        m = re.search(r"\bv_mfma_\S+\s+(v\[\d+:\d+\])", line)
        if not m:
            continue
        dst = _regs(m.group(1))
        slots = 0
        for k in range(i + 1, min(i + 200, len(lines))):
            t = lines[k].strip()
            if not t or t.startswith(";") or t.endswith(":") or t.startswith("."):
                continue                      # labels fall through
            op = t.split(None, 1)[0]
            if op in ("s_branch", "s_endpgm", "s_setpc_b64"):
                break                         # leaves the fall-through path
            mm = re.match(r"s_nop (\d+)", t)
            if mm:
                slots += int(mm.group(1)) + 1
                continue
            args = t.split(None, 1)[1].split(",") if " " in t else []
            if op.startswith("v_mfma"):
                if _regs(",".join(args[1:])) & dst or _regs(args[0] if args else "") & dst:
                    break                     # chained MFMA: the hardware orders it
                slots += 1
                continue
            if op.startswith("v_") and _regs(",".join(args[1:])) & dst:
                if slots < MIN_SLOTS:
                    found.append((fn, k + 1, slots, t[:80]))
                break
            slots += 1
    return found


def test_mfma_results_are_not_read_too_soon(tmp_path):
    with cf.ThreadPoolExecutor(max_workers=len(SOURCES)) as ex:
        asms = dict(zip(SOURCES, ex.map(lambda s: _asm(s, str(tmp_path)), SOURCES)))
    problems = []
    for src, lines in asms.items():
        assert any("v_mfma" in l for l in lines), src
        problems += [(src,) + p for p in short_reads(lines)]
    assert not problems, "\n".join("%s %s line %d: %d slots before %s" % p for p in problems[:20])


def test_scanner_flags_a_short_read():
    # the pattern of the bug: MFMA, a branch, then a read of its result
    lines = ["_Zfn:", "\tv_mfma_f32_16x16x32_bf16 v[22:25], v[18:21], v[10:13], 0",
             "\ts_cbranch_vccz .LBB0_1", "\tv_min_i32_e32 v75, v22, v23"]
    assert short_reads(lines) and short_reads(lines)[0][2] == 1
    ok = ["_Zfn:", "\tv_mfma_f32_16x16x32_bf16 v[22:25], v[18:21], v[10:13], 0",
          "\ts_nop 7", "\tv_min_i32_e32 v75, v22, v23"]
    assert not short_reads(ok)
