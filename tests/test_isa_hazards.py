"""Checks the built gfx950 code of the GEMM kernels for the wait states that
the inline-assembly direct loads (global_load_lds with an SGPR base) need and
that the compiler's hazard tracking does not provide: 5 states after a VALU
write of a base SGPR, 1 state after an M0 write. Disassembles the library's
own device code; needs no GPU."""
import os
import re
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
BUILD = os.path.join(ROOT, "paper_1805_08939_amd", "_build")
LLVM = "/opt/rocm/llvm/bin"
TOOLS = [os.path.join(LLVM, t) for t in ("llvm-objcopy", "clang-offload-bundler", "llvm-objdump")]


def _disassemble(obj, tmp_path):
    fat, code = tmp_path / "fatbin", tmp_path / "code"
    subprocess.run([TOOLS[0], f"--dump-section=.hip_fatbin={fat}", obj, str(tmp_path / "host.o")], check=True)
    subprocess.run([TOOLS[1], "--type=o", "--targets=hipv4-amdgcn-amd-amdhsa--gfx950", f"--input={fat}",
                    f"--output={code}", "--unbundle"], check=True)
    out = subprocess.run([TOOLS[2], "-d", "--mcpu=gfx950", str(code)], check=True, capture_output=True, text=True)
    return out.stdout.split("\n")


def _sgprs(tok):
    m = re.match(r"s\[(\d+):(\d+)\]$", tok)
    if m:
        return set(range(int(m.group(1)), int(m.group(2)) + 1))
    m = re.match(r"s(\d+)$", tok)
    return {int(m.group(1))} if m else set()


def hazards(lines):
    """(checked loads, list of violations) over a disassembly listing."""
    hist, bad, n = [], [], 0   # hist: (text, dst sgprs, writes m0, is valu, wait states)
    for ln in lines:
        if re.match(r"^[0-9a-f]+ <.*>:$", ln):
            hist = []
            continue
        t = ln.split("//")[0].strip()
        if not t or t.endswith(":"):
            continue
        op = t.split()[0]
        args = [a.strip() for a in t[len(op):].split(",")]
        if op.startswith("global_load_lds"):
            n += 1
            need = _sgprs(args[1]) if len(args) > 1 else set()
            ws, valu_ok, m0_ok = 0, not need, False
            for text, dst, m0, valu, w in reversed(hist):
                if not m0_ok and m0:
                    if ws < 1:
                        bad.append(f"M0 write '{text}' then '{t}' after {ws} wait states")
                    m0_ok = True
                if not valu_ok and valu and dst & need:
                    if ws < 5:
                        bad.append(f"VALU SGPR write '{text}' then '{t}' after {ws} wait states")
                    valu_ok = True
                ws += w
                if ws >= 5 and m0_ok:
                    break
        w = int(args[0], 0) + 1 if op == "s_nop" else 1
        dst = _sgprs(args[0]) if args and args[0] else set()
        hist.append((t, dst, bool(args and args[0] == "m0"), op.startswith("v_"), w))
        hist = hist[-40:]
    return n, bad


# every device source of the library; the first three hold direct-load kernels
SOURCES = ["ard_fc.hip", "ard_tile.hip", "ard_lstm.hip", "ard_lstm_tile.hip", "ard_dropout.hip"]
DIRECT_LOADS = {"ard_fc.hip", "ard_tile.hip", "ard_lstm.hip"}


def test_every_device_source_is_checked():
    assert sorted(SOURCES) == sorted(f for f in os.listdir(os.path.join(os.path.dirname(BUILD), "csrc"))
                                     if f.endswith(".hip"))


@pytest.mark.skipif(not all(os.path.exists(t) for t in TOOLS), reason="ROCm LLVM tools not found")
@pytest.mark.parametrize("src", SOURCES)
def test_direct_load_wait_states(tmp_path, src):
    obj = os.path.join(BUILD, src + ".o")
    if not os.path.exists(obj):
        pytest.skip("library objects not built")
    n, bad = hazards(_disassemble(obj, tmp_path))
    if src in DIRECT_LOADS:
        assert n > 0, f"no direct loads found in the kernels of {src}"
    assert not bad, "\n".join(bad[:10])


def test_checker_flags_a_short_gap():
    """The checker itself: a readfirstlane two states before the load is flagged,
    five states are enough."""
    short = ["0 <k>:", "\tv_readfirstlane_b32 s4, v1", "\ts_mov_b32 m0, s6", "\ts_nop 0",
             "\tglobal_load_lds_dwordx4 v2, s[4:5]"]
    ok = ["0 <k>:", "\tv_readfirstlane_b32 s4, v1", "\ts_mov_b32 m0, s6", "\ts_nop 3",
          "\tglobal_load_lds_dwordx4 v2, s[4:5]"]
    nomo = ["0 <k>:", "\ts_mov_b32 m0, s6", "\tglobal_load_lds_dwordx4 v2, s[4:5]"]
    assert len(hazards(short)[1]) == 1
    assert hazards(ok)[1] == []
    assert len(hazards(nomo)[1]) == 1


def _kernel_notes(obj, tmp_path):
    fat, code = tmp_path / "fatbin", tmp_path / "code"
    subprocess.run([TOOLS[0], f"--dump-section=.hip_fatbin={fat}", obj, str(tmp_path / "host.o")], check=True)
    subprocess.run([TOOLS[1], "--type=o", "--targets=hipv4-amdgcn-amd-amdhsa--gfx950", f"--input={fat}",
                    f"--output={code}", "--unbundle"], check=True)
    readobj = os.path.join(LLVM, "llvm-readobj")
    return subprocess.run([readobj, "--notes", str(code)], check=True, capture_output=True, text=True).stdout


@pytest.mark.skipif(not all(os.path.exists(t) for t in TOOLS + [os.path.join(LLVM, "llvm-readobj")]),
                    reason="ROCm LLVM tools not found")
@pytest.mark.parametrize("src", SOURCES)
def test_no_kernel_spills_registers(tmp_path, src):
    """A VGPR spill goes to scratch memory, and inside a GEMM main loop it
    costs more than the kernel's arithmetic: every kernel of the library must
    fit its vector registers (SGPR spills land in VGPR lanes and are cheap)."""
    obj = os.path.join(BUILD, src + ".o")
    if not os.path.exists(obj):
        pytest.skip("library objects not built")
    notes = _kernel_notes(obj, tmp_path)
    kernels = re.findall(r"\.name:\s+(\S+)(.*?)(?=\n  - |\Z)", notes, re.S)
    assert kernels, "no kernel metadata found"
    bad = []
    for name, body in kernels:
        m = re.search(r"\.vgpr_spill_count:\s+(\d+)", body)
        if m and int(m.group(1)) > 0:
            bad.append(f"{name}: vgpr_spill_count {m.group(1)}")
    assert not bad, "\n".join(bad)

