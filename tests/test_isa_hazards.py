"""Scan the gfx950 assembly of the library's kernels for a store-data hazard
(no GPU): a vector-memory store of more than 8 bytes must not be followed
directly by a VALU instruction that overwrites one of the store's data
registers.  The compiler guards this for most store forms, but not for
buffer stores whose scalar offset is a register, and a GPU run showed such a
store writing the overwritten value.  The kernels keep every buffer store's
scalar offset at the literal 0; this test keeps it that way."""
import os
import re
import subprocess

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ASM = os.path.join(ROOT, "_build", "kernels-gfx950.s")

STORE = re.compile(r"^\s*(buffer|global|flat|scratch)_store_dwordx([34])\s+(.*)$")
VREG = re.compile(r"v\[(\d+):(\d+)\]|v(\d+)\b")


def _regs(tok):
    m = VREG.fullmatch(tok.strip())
    if not m:
        return set()
    if m.group(3) is not None:
        return {int(m.group(3))}
    return set(range(int(m.group(1)), int(m.group(2)) + 1))


def _instructions(text):
    for line in text.splitlines():
        s = line.split(";")[0].strip()
        if not s or s.endswith(":") or s.startswith("."):
            continue
        yield s


def hazards(text):
    found = []
    ins = list(_instructions(text))
    for k, s in enumerate(ins[:-1]):
        m = STORE.match(s)
        if not m:
            continue
        ops = [o.strip() for o in m.group(3).split(",")]
        data = ops[0] if m.group(1) == "buffer" else ops[1]
        regs = _regs(data)
        nxt = ins[k + 1]
        if not nxt.startswith("v_"):
            continue
        parts = nxt.split(None, 1)
        if len(parts) < 2:
            continue
        dst = parts[1].split(",")[0]
        if regs & _regs(dst):
            found.append((s, nxt))
    return found


def test_scanner_sees_the_pattern():
    bad = "buffer_store_dwordx4 v[6:9], v1, s[48:51], s33 offen nt\n\tv_xor_b32_e32 v6, v10, v9\n"
    good = "buffer_store_dwordx4 v[6:9], v1, s[48:51], 0 offen nt\n\ts_nop 0\n\tv_xor_b32_e32 v6, v10, v9\n"
    assert hazards(bad) and not hazards(good)
    assert not hazards("global_store_dwordx2 v[0:1], v[6:7], off\n\tv_mov_b32 v6, 0\n")


def test_library_kernels_have_no_store_data_hazard():
    subprocess.run(["make", "-s", "-C", ROOT, "isa"], check=True)
    text = open(ASM).read()
    assert "buffer_store_dwordx4" in text
    found = hazards(text)
    assert not found, found[:5]
    # and no buffer store carries a register scalar offset
    for line in _instructions(text):
        if line.startswith("buffer_store"):
            ops = [o.strip() for o in line.split(None, 1)[1].split(",")]
            assert not ops[3].startswith("s"), line
