"""Store-data hazard check on the built library's own gfx950 code (no GPU needed).

On this part a vector-memory store of more than 8 bytes reads its data registers after it
issues; an instruction that rewrote those registers 1-3 instructions after a 16-byte store
corrupted the stored values (seen on the G kernel's epilogue), although the compiler only keeps
one wait state there. The built code object is extracted from liblce.so and disassembled, and
no instruction among the MIN_GAP - 1 that follow such a store (an s_nop N counting as N + 1)
may write one of its data registers. Stores that would break this are written with
store16_padded (the store and 8 wait states in one statement).
"""
import os
import re
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIB = os.path.join(ROOT, "paper_2605_21442_amd", "liblce.so")
LLVM = "/opt/rocm/llvm/bin"
MIN_GAP = 8

STORE = re.compile(r"^(buffer_store_dwordx[34]|global_store_dwordx[34]|flat_store_dwordx[34])\s+(.*)$")
VREG = re.compile(r"v\[(\d+):(\d+)\]|v(\d+)\b")
NO_VGPR_DST = ("v_cmp", "v_readlane", "v_readfirstlane", "s_", "buffer_store", "global_store", "flat_store",
               "ds_write", "ds_bpermute", "scratch_store")


def _regs(tok):
    m = VREG.match(tok.strip())
    if not m:
        return None
    if m.group(1):
        return int(m.group(1)), int(m.group(2))
    return int(m.group(3)), int(m.group(3))


def _disassemble(tmp):
    fat, co = os.path.join(tmp, "fat.bin"), os.path.join(tmp, "dev.co")
    subprocess.run([f"{LLVM}/llvm-objcopy", "--dump-section", f".hip_fatbin={fat}", LIB], check=True)
    subprocess.run([f"{LLVM}/clang-offload-bundler", "--unbundle", "--type=o", f"--input={fat}",
                    "--targets=hipv4-amdgcn-amd-amdhsa--gfx950", f"--output={co}"], check=True)
    out = subprocess.run([f"{LLVM}/llvm-objdump", "-d", "--mcpu=gfx950", co], check=True, capture_output=True,
                         text=True).stdout
    return out.splitlines()


def violations(lines):
    """(function, store, writer, gap) for each wide store whose data registers are written again
    fewer than MIN_GAP wait states after it."""
    func, bad = None, []
    for i, l in enumerate(lines):
        if l.endswith(">:"):
            func = l
            continue
        m = STORE.match(l)
        if not m:
            continue
        ops = [t.strip() for t in m.group(2).split(",")]
        data = _regs(ops[0] if m.group(1).startswith("buffer") else ops[1])
        if data is None:
            continue
        lo, hi = data
        n = 0
        for k in range(i + 1, len(lines)):
            y = lines[k]
            if y.endswith(">:") or y.startswith("s_endpgm"):
                break   # (after s_endpgm the wave runs nothing more; what follows is another block)
            if not y:
                continue
            nop = re.match(r"s_nop\s+(0x[0-9a-fA-F]+|\d+)", y)
            n += (int(nop.group(1), 0) + 1) if nop else 1   # s_nop N gives N + 1 wait states
            if n >= MIN_GAP:
                break
            if y.startswith(NO_VGPR_DST):
                continue
            parts = y.split(None, 1)
            if len(parts) < 2:
                continue
            dst = _regs(parts[1].split(",")[0])
            if dst and dst[0] <= hi and dst[1] >= lo:
                bad.append((func, l, y, n))
                break
    return bad


def test_scanner_flags_short_gaps_only():
    lines = ["<k>:", "buffer_store_dwordx4 v[4:7], v0, s[0:3], 0 offen", "v_mov_b32_e32 v1, v2",
             "v_mul_f32_e32 v5, v6, v7",                                   # rewrites v5: 2 after
             "global_store_dwordx4 v[8:9], v[10:13], off", "s_nop 7", "v_mov_b32_e32 v10, 0",   # 9 after
             "global_store_dwordx2 v[8:9], v[20:21], off", "v_mov_b32_e32 v20, 0",              # 8 bytes
             "buffer_store_dwordx4 v[4:7], v0, s[0:3], 0 offen", "s_endpgm", "v_mov_b32_e32 v5, 0"]  # wave ended
    bad = violations(lines)
    assert [(b[1].split()[0], b[3]) for b in bad] == [("buffer_store_dwordx4", 2)]


def test_no_store_data_rewritten_right_after_a_wide_store(tmp_path):
    if not os.path.exists(LIB) or not all(shutil.which(f"{LLVM}/{t}") for t in
                                          ("llvm-objcopy", "clang-offload-bundler", "llvm-objdump")):
        pytest.skip("built library or ROCm LLVM tools missing")
    lines = [l.split("//")[0].strip() for l in _disassemble(str(tmp_path))]
    assert sum(1 for l in lines if STORE.match(l)) > 0
    bad = violations(lines)
    assert not bad, "\n".join(f"{f} {st} ... {w} ({n} after)" for f, st, w, n in bad)
