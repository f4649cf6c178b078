"""Built-code check of the kernels' inline-asm LDS reads (CPU, needs hipcc).

Some staged reads are issued by one inline-asm statement and waited for by a
later one (s_waitcnt lgkmcnt), so that the wait can overlap other work.  The
compiler does not know the read is still in flight and may not touch its
destination registers in between: a copy or use before the wait would read
stale data.  This test compiles the kernel sources to gfx950 assembly and
checks, for every inline-asm LDS read, that no instruction reads or writes its
destination registers before an s_waitcnt lgkmcnt that retires it.  A planted
hazard in a synthetic listing checks the scanner itself.
"""
import os
import re
import shutil
import subprocess

import pytest

from paper_2506_20686_amd import build as hipbuild

HIPCC = hipbuild.HIPCC
CSRC = hipbuild.CSRC
SOURCES = ("fwd.hip", "bwd.hip", "lnl.hip", "trn.hip")

needs_hipcc = pytest.mark.skipif(not (os.path.exists(HIPCC) or shutil.which("hipcc")),
                                 reason="hipcc not available")


def _regs(tok):
    m = re.match(r"v\[(\d+):(\d+)\]", tok)
    if m:
        return set(range(int(m.group(1)), int(m.group(2)) + 1))
    m = re.match(r"v(\d+)$", tok)
    return {int(m.group(1))} if m else set()


def scan(text):
    """(inline-asm LDS reads checked, [hazard descriptions])."""
    checked, bad = 0, []
    kern, in_asm, pending = None, False, []  # pending: [regs, line, LDS ops issued after]
    for i, line in enumerate(text.splitlines()):
        if re.match(r"^_Z\w+:", line):
            kern, pending = line.split(":")[0], []
        if ";;#ASMSTART" in line:
            in_asm = True
            continue
        if ";;#ASMEND" in line:
            in_asm = False
            continue
        body = line.split(";")[0].strip()
        if not body or body.startswith(".") or body.endswith(":"):
            continue
        parts = body.split(None, 1)
        op = parts[0]
        ops = [t.strip() for t in parts[1].split(",")] if len(parts) > 1 else []
        if op == "s_waitcnt":
            m = re.search(r"lgkmcnt\((\d+)\)", body)
            if m:
                n = int(m.group(1))
                pending = [p for p in pending if p[2] < n] if n > 0 else []
            continue
        if in_asm and op in ("ds_read_b64_tr_b16", "ds_read_b128"):
            checked += 1
            pending = [[r, ln, c + 1] for r, ln, c in pending]
            pending.append([_regs(ops[0]), i, 0])
            continue
        if op.startswith("ds_") or op.startswith("s_load") or op.startswith("s_buffer_load"):
            pending = [[r, ln, c + 1] for r, ln, c in pending]
        used = set()
        for t in ops:
            used |= _regs(t)
        for r, ln, _ in pending:
            if used & r:
                bad.append(f"{kern}: line {i + 1} '{body}' touches a read of line {ln + 1}")
    return checked, bad


def test_scanner_finds_a_planted_hazard():
    text = "\n".join([
        "_Zk:",
        "\t;;#ASMSTART", "\tds_read_b64_tr_b16 v[10:11], v2 offset:0", "\t;;#ASMEND",
        "\tv_mov_b32_e32 v20, v11",            # before the wait: a hazard
        "\ts_waitcnt lgkmcnt(0)",
        "\t;;#ASMSTART", "\tds_read_b64_tr_b16 v[12:13], v2 offset:64", "\t;;#ASMEND",
        "\tds_read_b128 v[30:33], v3",
        "\ts_waitcnt lgkmcnt(1)",              # retires the older read
        "\tv_add_f32_e32 v40, v12, v12",
    ])
    checked, bad = scan(text)
    assert checked == 2 and len(bad) == 1 and "v_mov_b32_e32 v20, v11" in bad[0]


@needs_hipcc
@pytest.mark.parametrize("src", SOURCES)
def test_no_use_of_a_pending_lds_read(tmp_path, src):
    out = tmp_path / (src + ".s")
    cmd = [HIPCC, "--offload-arch=gfx950", "-O3", "-std=c++17", "--cuda-device-only", "-S",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-Xarch_device", "-fno-honor-nans",
           "-I", os.path.join(hipbuild.ROOT, "include"), "-I", CSRC,
           os.path.join(CSRC, src), "-o", str(out)]
    res = subprocess.run(cmd, capture_output=True, text=True)
    assert res.returncode == 0, res.stderr[-2000:]
    checked, bad = scan(out.read_text())
    assert checked > 0, "no inline-asm LDS reads found: the scan is not looking at them"
    assert not bad, "\n".join(bad[:20])
