"""Static check of the compiled kernels: no 16-byte (or 12-byte) vector-memory store may have its data registers
overwritten by one of the next two instructions.

On gfx950 a buffer store of 16 bytes with a register offset was seen to write values that the very next VALU
instruction put into its data registers; the compiler inserts no wait state there.  The row kernel's grouped
dlogits stores therefore carry two wait states each.  This test compiles every kernel source to gfx950 assembly
(no GPU needed) and fails if any store in the library is followed that closely by a write to its data registers,
so a change of code or compiler that brings the pattern back is caught before it runs.

Two more checks of the same assembly.  The packed-operand GEMM core loads B fragments with inline asm, which the
compiler cannot count: no instruction may write a register that such a load is still filling before a
vmcnt(0) wait (a late load would overwrite it; an index overwritten this way once sent a load to a wild
address).  And the token-blocked schedule runs its D pass beside the forward product on every CU, which needs
both workgroups' registers and LDS to fit one CU together.
"""
import functools
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


def _instructions(asm: str) -> list:
    fn, insts = None, []
    for line in asm.splitlines():
        if re.match(r"^[_A-Za-z][\w.$]*:", line) and not line.startswith(".L"):
            fn = line.split(":")[0]
        s = line.split(";")[0].strip()
        if s and not s.startswith(".") and not s.endswith(":"):
            insts.append((fn, s))
    return insts


def scan_late_loads(asm: str) -> list:
    """(function, load, offending instruction) for every 16-byte buffer load into registers (not into LDS) whose
    destination a later instruction of the same function writes before a vmcnt(0) wait, in program order (which
    also covers the path out of a loop after its last iteration)."""
    insts, hits = _instructions(asm), []
    for i, (fn, s) in enumerate(insts):
        op = s.split()[0]
        if op != "buffer_load_dwordx4" or s.endswith(" lds"):
            continue
        dst = _vregs(s[len(op):].split(",")[0].strip())
        for fn2, s2 in insts[i + 1:]:
            op2 = s2.split()[0]
            if fn2 != fn or op2 == "s_endpgm" or (op2 == "s_waitcnt" and "vmcnt(0)" in s2):
                break
            if not op2.startswith(("v_", "ds_read", "global_load", "buffer_load", "flat_load", "scratch_load")):
                continue
            if op2.startswith(("v_cmp", "v_readlane", "v_readfirstlane")):
                continue
            if _vregs(s2[len(op2):].split(",")[0].strip()) & dst:
                if not op2.startswith("buffer_load"):  # the next load into the same registers is fine
                    hits.append((fn, s, s2))
                break
    return hits


def test_late_load_scanner_finds_the_pattern():
    bad = ("k:\n\tbuffer_load_dwordx4 v[130:133], v192, s[8:11], 0 offen\n\ts_add_i32 s4, s4, 1\n"
           "\tv_and_b32_e32 v130, 0xc0, v0\n\ts_waitcnt vmcnt(0)\n")
    assert len(scan_late_loads(bad)) == 1
    ok = ("k:\n\tbuffer_load_dwordx4 v[130:133], v192, s[8:11], 0 offen\n\ts_waitcnt vmcnt(0)\n"
          "\tv_and_b32_e32 v130, 0xc0, v0\n")
    lds = "k:\n\tbuffer_load_dwordx4 v9, s[12:15], 0 offen lds\n\tv_mov_b32_e32 v9, 0\n"
    assert scan_late_loads(ok) == [] and scan_late_loads(lds) == []


SOURCES = sorted(f for f in os.listdir(CSRC) if f.endswith(".hip")) + ["bench/stream_copy.hip"]


@functools.lru_cache(maxsize=None)
def _assembly(src: str) -> str:
    import tempfile
    d = tempfile.mkdtemp()
    out = os.path.join(d, os.path.basename(src) + ".s")
    cmd = [HIPCC, "--offload-arch=gfx950", "-O3", "-std=c++17", "-Xclang", "-target-feature", "-Xclang",
           "-packed-fp32-ops", "-I" + os.path.join(ROOT, "include"), "-I" + CSRC, "--cuda-device-only", "-S",
           os.path.join(CSRC, src), "-o", out]
    subprocess.run(cmd, check=True, capture_output=True)
    with open(out) as f:
        text = f.read()
    shutil.rmtree(d, ignore_errors=True)
    return text


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not installed")
@pytest.mark.parametrize("src", SOURCES)
def test_no_store_data_overwrite(src):
    hits = scan(_assembly(src))
    assert not hits, "\n".join(f"{fn}: [{a}] then [{b}]" for fn, a, b in hits[:10])


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not installed")
@pytest.mark.parametrize("src", SOURCES)
def test_no_register_reuse_under_a_late_load(src):
    hits = scan_late_loads(_assembly(src))
    assert not hits, "\n".join(f"{fn}: [{a}] then [{b}]" for fn, a, b in hits[:10])


def _kernel_resources(asm: str) -> dict:
    res = {}
    for block in asm.split("  - .agpr_count:")[1:]:
        name = re.search(r"\.name:\s+(\S+)", block).group(1)
        res[name] = dict(vgpr=int(re.search(r"\.vgpr_count:\s+(\d+)", block).group(1)),
                         lds=int(re.search(r"\.group_segment_fixed_size:\s+(\d+)", block).group(1)),
                         spill=int(re.search(r"\.vgpr_spill_count:\s+(\d+)", block).group(1)))
    return res


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not installed")
def test_d_pass_fits_beside_the_forward_product():
    """One forward-product workgroup (8 waves, two per SIMD) and one D-pass workgroup (4 waves, one per SIMD) on
    one CU: 512 registers per lane per SIMD, allocated 8 at a time, and 160 KB of LDS."""
    res = _kernel_resources(_assembly("lmhead.hip"))
    # the token-blocked forward product: k_lm_partial<STORE_Z = false, PACKED = true, TERMS = true>
    fwd = [v for k, v in res.items() if k.startswith("_ZN4grpo12k_lm_partialILb0ELb1ELb1E")]
    dpass = [v for k, v in res.items() if k.startswith("_ZN4grpo14k_lm_block_d16")]
    assert len(fwd) == 1 and len(dpass) == 1, sorted(res)
    alloc = lambda n: (n + 7) // 8 * 8
    assert 2 * alloc(fwd[0]["vgpr"]) + alloc(dpass[0]["vgpr"]) <= 512, (fwd, dpass)
    assert fwd[0]["lds"] + dpass[0]["lds"] <= 160 * 1024, (fwd, dpass)
    assert fwd[0]["spill"] == 0 and dpass[0]["spill"] == 0
