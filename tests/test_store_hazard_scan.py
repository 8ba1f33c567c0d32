"""Static check of the compiled kernels: no 16-byte (or 12-byte) vector-memory store may have its data registers
overwritten by one of the next two instructions.

On gfx950 a buffer store of 16 bytes with a register offset was seen to write values that the very next VALU
instruction put into its data registers; the compiler inserts no wait state there.  The row kernel's grouped
dlogits stores therefore carry two wait states each.  This test compiles every kernel source to gfx950 assembly
(no GPU needed) and fails if any store in the library is followed that closely by a write to its data registers,
so a change of code or compiler that brings the pattern back is caught before it runs.
"""
import os
import re
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2606_05597_amd", "csrc")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
WINDOW = 2  # instructions after the store that must not write its data registers

STORE = re.compile(r"^(buffer|global|flat|scratch)_store_(dwordx3|dwordx4|b96|b128)$")


def _vregs(tok: str) -> set:
    m = re.fullmatch(r"v\[(\d+):(\d+)\]", tok)
    if m:
        return set(range(int(m.group(1)), int(m.group(2)) + 1))
    m = re.fullmatch(r"v(\d+)", tok)
    return {int(m.group(1))} if m else set()


def scan(asm: str) -> list:
    """(function, store, offending instruction) for every store whose data registers one of the next WINDOW
    instructions writes (VALU destinations; loads return later and are not counted)."""
    fn, insts, hits = None, [], []
    for line in asm.splitlines():
        if re.match(r"^[_A-Za-z][\w.$]*:", line) and not line.startswith(".L"):
            fn = line.split(":")[0]
        s = line.split(";")[0].strip()
        if not s or s.startswith(".") or s.endswith(":"):
            continue
        insts.append((fn, s))
    for i, (fn, s) in enumerate(insts):
        op = s.split()[0]
        if not STORE.match(op):
            continue
        ops = [o.strip() for o in s[len(op):].split(",")]
        data = _vregs(ops[0] if op.startswith(("buffer", "scratch")) else ops[1])
        for k in range(1, WINDOW + 1):
            if i + k >= len(insts):
                break
            s2 = insts[i + k][1]
            op2 = s2.split()[0]
            if op2 == "s_nop":
                break  # wait states: the store has read its data
            if not op2.startswith("v_") or op2.startswith(("v_cmp", "v_readlane", "v_readfirstlane")):
                continue
            if _vregs(s2[len(op2):].split(",")[0].strip()) & data:
                hits.append((fn, s, s2))
    return hits


def test_scanner_finds_the_pattern():
    bad = "k:\n\tbuffer_store_dwordx4 v[58:61], v101, s[56:59], s93 offen nt\n\tv_lshlrev_b32_e32 v58, 16, v54\n"
    assert len(scan(bad)) == 1
    ok_nop = "k:\n\tbuffer_store_dwordx4 v[58:61], v101, s[56:59], s93 offen nt\n\ts_nop 1\n\tv_mov_b32_e32 v58, 0\n"
    ok_load = "k:\n\tbuffer_store_dwordx4 v[58:61], v101, s[56:59], s93 offen nt\n\tbuffer_load_dwordx4 v[58:61], v101, s[60:63], s93 offen nt\n"
    ok_far = "k:\n\tglobal_store_dwordx4 v1, v[8:11], s[0:1]\n\tv_add_u32_e32 v2, 1, v2\n\ts_add_i32 s3, s3, 1\n\tv_mov_b32_e32 v8, 0\n"
    assert scan(ok_nop) == [] and scan(ok_load) == [] and scan(ok_far) == []


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not installed")
@pytest.mark.parametrize("src", sorted(f for f in os.listdir(CSRC) if f.endswith(".hip")) + ["bench/stream_copy.hip"])
def test_no_store_data_overwrite(src, tmp_path):
    out = tmp_path / (os.path.basename(src) + ".s")
    cmd = [HIPCC, "--offload-arch=gfx950", "-O3", "-std=c++17", "-Xclang", "-target-feature", "-Xclang",
           "-packed-fp32-ops", "-I" + os.path.join(ROOT, "include"), "-I" + CSRC, "--cuda-device-only", "-S",
           os.path.join(CSRC, src), "-o", str(out)]
    subprocess.run(cmd, check=True, capture_output=True)
    hits = scan(out.read_text())
    assert not hits, "\n".join(f"{fn}: [{a}] then [{b}]" for fn, a, b in hits[:10])
    shutil.rmtree(tmp_path, ignore_errors=True)
