"""Host-side check of the device code the compiler generates from this
repository's kernels (no GPU needed; skipped when hipcc is absent).

A vector-memory store of more than 8 bytes reads its data registers after
issue; a VALU instruction that overwrites them in the very next slot can
change the stored value.  The compiler inserts the wait state for buffer
stores only when their scalar offset is not a register, so every buffer store
here takes a zero scalar offset (the offset goes into the vector offset).
Measured on gfx950: with a register scalar offset the loss-only kernel stored
small integers (the next chunk's address) in place of a few d_logits values,
differently from run to run.  This test keeps both rules in the assembly."""
import os
import re
import shutil
import subprocess

import pytest

from paper_2505_17826_amd import build_lib as B

HIPCC = B.HIPCC if os.path.exists(B.HIPCC) else shutil.which("hipcc")
pytestmark = pytest.mark.skipif(not HIPCC, reason="hipcc not available")


def _sources_with_stores():
    """Every device source: besides the explicit buffer stores, plain 16-byte
    assignments compile to wide global stores, and the next-slot rule holds
    for those too."""
    return list(B.SOURCES)


def _vregs(tok):
    m = re.match(r"v\[(\d+):(\d+)\]", tok)
    if m:
        return set(range(int(m.group(1)), int(m.group(2)) + 1))
    m = re.match(r"v(\d+)$", tok)
    return {int(m.group(1))} if m else set()


def _check_asm(asm):
    """(stores with a register scalar offset, stores whose data the next
    instruction overwrites), as lists of (store, next) lines."""
    reg_soff, overwritten = [], []
    prev = None
    for line in asm.splitlines():
        s = line.strip()
        if not s or s[0] in ";." or s.endswith(":"):
            continue
        ops = [o for o in re.split(r"[\s,]+", s) if o]
        if prev is not None:
            if ops[0].startswith("v_") and len(ops) > 1 and _vregs(ops[1]) & prev[1]:
                overwritten.append((prev[0], s))
            prev = None
        m = re.match(r"(buffer|global|flat)_store_dwordx([34])$", ops[0])
        if m:
            data = _vregs(ops[1] if m.group(1) == "buffer" else ops[2])
            if m.group(1) == "buffer" and re.match(r"s\d+$", ops[4]):
                reg_soff.append((s, ""))
            prev = (s, data)
    return reg_soff, overwritten


def test_checker_flags_the_pattern():
    bad = ("buffer_store_dwordx4 v[10:13], v14, s[4:7], s3 offen nt\n"
           "v_or_b32_e32 v10, 0x400, v0\n")
    good = ("buffer_store_dwordx4 v[10:13], v14, s[4:7], 0 offen nt\n"
            "s_nop 0\n"
            "v_or_b32_e32 v10, 0x400, v0\n")
    r, o = _check_asm(bad)
    assert len(r) == 1 and len(o) == 1
    assert _check_asm(good) == ([], [])


@pytest.mark.parametrize("src", _sources_with_stores())
def test_wide_stores_are_protected(src, tmp_path):
    out = tmp_path / (src + ".s")
    cmd = [HIPCC, *[f for f in B.CFLAGS if f != "-fPIC"], *B.SOURCE_FLAGS.get(src, []),
           "--cuda-device-only", "-S", os.path.join(B.CSRC, src), "-o", str(out)]
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, r.stderr[-2000:]
    reg_soff, overwritten = _check_asm(out.read_text())
    assert not reg_soff, f"buffer stores with a register scalar offset: {reg_soff[:3]}"
    assert not overwritten, f"store data overwritten in the next slot: {overwritten[:3]}"
