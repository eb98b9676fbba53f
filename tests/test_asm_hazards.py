"""The gfx950 device code has no unprotected SGPR hazard in front of a buffer instruction (CPU only).

A buffer instruction that reads an SGPR (its resource, or M0 for an LDS DMA) needs 5 wait
states after a VALU instruction wrote that SGPR (v_readfirstlane, v_readlane when the compiler
reloads a spilled SGPR, a VALU compare or carry-out).  The compiler inserts them for the loads
it emits itself, but not in front of inline asm, so the GEMM's LDS-DMA asm carries its own.
Without them the load can use the register's previous value: a wrong base or format, and a
wrong operand tile.  Each kernel source is compiled to device assembly and scanned.
"""

import concurrent.futures
import os
import re
import subprocess
import tempfile

import pytest

from paper_2511_02302_amd import build as ff8_build

_VALU_SGPR_DEF = re.compile(
    r"^(v_readlane_b32|v_readfirstlane_b32|v_cmpx?_\w+|v_(?:add|sub|subrev|addc|subb|subbrev)_co\w*|"
    r"v_div_scale\w*|v_mad_[iu]64_[iu]32)\s+(\S+?),")
_WAIT_STATES = 5


def _sgprs(tok):
    tok = tok.strip()
    if tok == "m0":
        return {"m0"}
    if tok in ("vcc", "vcc_lo", "vcc_hi"):
        return {"vcc"}
    m = re.fullmatch(r"s(\d+)", tok)
    if m:
        return {int(m.group(1))}
    m = re.fullmatch(r"s\[(\d+):(\d+)\]", tok)
    if m:
        return set(range(int(m.group(1)), int(m.group(2)) + 1))
    return set()


def hazards(asm_text):
    """(VALU def, buffer instruction, wait states between) for each buffer instruction that
    reads an SGPR written by a VALU instruction fewer than 5 wait states before it on the
    straight-line path (labels are passed, unconditional branches end the walk; s_nop N
    counts N + 1 wait states, any other instruction 1)."""
    lines = []
    for raw in asm_text.splitlines():
        s = raw.split(";")[0].strip()
        if s and not s.startswith(".") and not s.endswith(":"):
            lines.append(s)
    found = []
    for i, ins in enumerate(lines):
        if not ins.startswith("buffer_"):
            continue
        parts = ins.split(None, 1)
        ops = [o.strip() for o in parts[1].split(",")] if len(parts) > 1 else []
        uses = set().union(*(_sgprs(o) for o in ops)) if ops else set()
        if re.search(r"\blds\b", ins):
            uses.add("m0")
        ws = 0
        for j in range(i - 1, -1, -1):
            prev = lines[j]
            if ws >= _WAIT_STATES or prev.startswith(("s_branch", "s_setpc", "s_endpgm")):
                break
            if prev.startswith("s_nop"):
                ws += int(prev.split()[1], 0) + 1
                continue
            m = _VALU_SGPR_DEF.match(prev)
            if m and _sgprs(m.group(2)) & uses:
                found.append((prev, ins, ws))
                break
            ws += 1
    return found


def test_scanner_finds_a_planted_hazard():
    bad = "v_readlane_b32 s99, v172, 31\n\ts_nop 0\n\tbuffer_load_dwordx4 v24, s[96:99], 0 offen lds\n"
    assert len(hazards(bad)) == 1
    m0 = "v_readfirstlane_b32 m0, v3\n\ts_nop 1\n\tbuffer_load_dword v2, s[4:7], 0 offen lds\n"
    assert len(hazards(m0)) == 1
    ok = "v_readlane_b32 s99, v172, 31\n\ts_nop 4\n\tbuffer_load_dwordx4 v24, s[96:99], 0 offen lds\n"
    assert hazards(ok) == []
    unrelated = "v_readlane_b32 s50, v172, 31\n\tbuffer_load_dwordx4 v24, s[96:99], 0 offen lds\n"
    assert hazards(unrelated) == []
    spaced = ("v_readfirstlane_b32 s98, v1\n\ts_mov_b32 s3, 0\n\ts_add_i32 s4, s4, 1\n\ts_nop 2\n"
              "\tbuffer_load_dword v2, s[96:99], 0 offen\n")
    assert hazards(spaced) == []


def _device_asm(src, out_dir):
    out = os.path.join(out_dir, os.path.basename(src) + ".s")
    cmd = [ff8_build.hipcc()] + ff8_build.COMMON + ["-x", "hip", "--cuda-device-only", "-S", src, "-o", out]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"{' '.join(cmd)}\n{r.stderr}")
    return src, open(out).read()


def test_device_code_has_no_sgpr_hazard_before_buffer_loads():
    try:
        ff8_build.hipcc()
    except RuntimeError:
        pytest.skip("hipcc not available")
    srcs = [s for s in ff8_build.sources() if s.endswith(".hip")]
    with tempfile.TemporaryDirectory() as d, concurrent.futures.ThreadPoolExecutor(max_workers=4) as ex:
        results = list(ex.map(lambda s: _device_asm(s, d), srcs))
    n_lds_dma = 0
    for src, text in results:
        assert not hazards(text), (os.path.basename(src), hazards(text)[:5])
        n_lds_dma += len(re.findall(r"buffer_load_dword\w* [^\n]*\blds\b", text))
    assert n_lds_dma > 0  # the scan saw the GEMM's LDS DMA
