"""The built library's gfx950 code holds no 12- or 16-byte store whose data
registers the very next instruction overwrites by a vector ALU write.

Such a pair was seen on the GPU to write the ALU result in place of the
stored data (a buffer_store_dwordx4 with an SGPR soffset followed by a VALU
write of its first data register); the compiler inserts no wait state there.
The kernels avoid it by passing 16-byte buffer stores a zero soffset, for
which the compiler separates the two.  This test disassembles the code
objects of libhla.so (built here from this repository's sources) and checks
every store.  CPU only.
"""
import os
import re
import shutil
import struct
import subprocess
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIB = os.path.join(ROOT, "paper_2510_27258_amd", "libhla.so")
OBJDUMP = "/opt/rocm/llvm/bin/llvm-objdump"
MAGIC = b"__CLANG_OFFLOAD_BUNDLE__"
STORE = re.compile(r"^(buffer|global|scratch|flat)_store_dword(x3|x4)\b")


def _gfx950_code_objects(path):
    """The gfx950 entries of every clang offload bundle in the library."""
    data = open(path, "rb").read()
    pos = 0
    while True:
        i = data.find(MAGIC, pos)
        if i < 0:
            return
        n = struct.unpack_from("<Q", data, i + len(MAGIC))[0]
        p = i + len(MAGIC) + 8
        for _ in range(n):
            off, size, tlen = struct.unpack_from("<QQQ", data, p)
            p += 24
            triple = data[p:p + tlen].decode()
            p += tlen
            if triple.endswith("gfx950"):
                yield data[i + off:i + off + size]
        pos = i + len(MAGIC)


def _regs(tok):
    """Register file letter and indices of one operand (v5, v[4:7], a[0:3])."""
    m = re.match(r"([va])\[(\d+):(\d+)\]$", tok)
    if m:
        return {(m.group(1), r) for r in range(int(m.group(2)), int(m.group(3)) + 1)}
    m = re.match(r"([va])(\d+)$", tok)
    return {(m.group(1), int(m.group(2)))} if m else set()


def _instructions(text):
    for line in text.splitlines():
        line = line.split("//")[0].strip()
        if not line or line.endswith(":") or line.startswith((";", ".")) or "file format" in line:
            continue
        if line.startswith("Disassembly of"):
            continue
        yield line


def find_hazards(text):
    """(store, next) pairs where next is a VALU instruction writing a data
    register of a 12/16-byte store."""
    insts = list(_instructions(text))
    found = []
    for k, inst in enumerate(insts[:-1]):
        op = inst.split()[0]
        if not STORE.match(op):
            continue
        ops = [t for t in re.split(r"[\s,]+", inst)[1:] if t]
        data = _regs(ops[0] if op.startswith("buffer") else ops[1])
        nxt = insts[k + 1]
        nop = nxt.split()[0]
        if not nop.startswith("v_") or nop.startswith(("v_cmp_", "v_cmpx_")):
            continue
        dst = _regs(re.split(r"[\s,]+", nxt)[1])
        if dst & data:
            found.append((inst, nxt))
    return found


def test_detector_flags_the_observed_pair():
    text = ("\tbuffer_store_dwordx4 v[22:25], v137, s[4:7], s42 offen nt\n"
            "\tv_lshlrev_b32_e32 v22, 2, v85\n"
            "\tbuffer_store_dwordx4 v[2:5], v1, s[4:7], 0 offen\n"
            "\ts_nop 0\n"
            "\tv_mov_b32_e32 v2, 0\n"
            "\tglobal_store_dwordx4 v[6:7], v[0:3], off\n"
            "\tv_add_u32_e32 v6, 4, v6\n")
    hz = find_hazards(text)
    assert len(hz) == 1 and hz[0][1].startswith("v_lshlrev_b32_e32 v22")


@pytest.mark.skipif(not os.path.exists(LIB), reason="libhla.so is not built")
@pytest.mark.skipif(not os.path.exists(OBJDUMP), reason="llvm-objdump is not installed")
def test_library_has_no_store_data_hazard():
    tmp = tempfile.mkdtemp()
    try:
        hazards, n = [], 0
        for k, blob in enumerate(_gfx950_code_objects(LIB)):
            path = os.path.join(tmp, f"co{k}.o")
            open(path, "wb").write(blob)
            text = subprocess.run([OBJDUMP, "-d", path], capture_output=True, text=True, check=True).stdout
            n += 1
            hazards += find_hazards(text)
        assert n > 0, "no gfx950 code object found in libhla.so"
        assert not hazards, "\n".join(f"{a}  ->  {b}" for a, b in hazards[:10])
    finally:
        shutil.rmtree(tmp)
