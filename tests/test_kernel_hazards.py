"""CPU check of the gfx950 assembly of every kernel: no hand-written
instruction can sit inside a hazard window that the compiler does not see.

gfx950 needs wait states that the hardware does not enforce -- between a VALU
write of a VGPR and a v_permlane16/32_swap reading it, between an MFMA and a
VALU read of its result, between an SALU write of M0 and an LDS DMA reading
it.  The compiler's hazard recognizer inserts them only around instructions it
sees; inline assembly is opaque to it.  So the kernels keep every VALU
instruction out of inline assembly (the permlane swaps and maxima are
builtins), and the one asm form left, the LDS DMA, carries its own M0 wait
state.  The device code is compiled to assembly here (no GPU) and read."""
import os
import re
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2607_02640_amd", "csrc")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
SOURCES = ["mtn_kernels.hip", "mtn_mfma.hip"]
REG = re.compile(r"\bv(?:\[(\d+):(\d+)\]|(\d+)\b)")


def _asm(src, out_dir):
    """The gfx950 assembly of `src`, built with the library's own options."""
    sys.path.insert(0, ROOT)
    from paper_2607_02640_amd import build
    out = os.path.join(out_dir, src + ".s")
    cmd = [HIPCC, *build.compile_flags(src), "--cuda-device-only", "-S", os.path.join(CSRC, src),
           "-o", out]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-3000:]
    return out


@pytest.fixture(scope="module")
def listings(tmp_path_factory):
    if not os.path.exists(HIPCC):
        pytest.skip("hipcc not available")
    d = str(tmp_path_factory.mktemp("asm"))
    with ThreadPoolExecutor(len(SOURCES)) as ex:
        paths = list(ex.map(lambda s: _asm(s, d), SOURCES))
    return {s: open(p).read().splitlines() for s, p in zip(SOURCES, paths)}


def _instructions(lines):
    """(mnemonic, operands, inside_inline_asm) per instruction, labels and
    directives dropped; a label ends the linear run (None marks it)."""
    out, in_asm = [], False
    for raw in lines:
        s = raw.strip()
        if s.startswith(";;#ASMSTART"):
            in_asm = True
            continue
        if s.startswith(";;#ASMEND"):
            in_asm = False
            continue
        s = s.split(";")[0].strip()
        if not s or s.startswith("."):
            continue
        if s.endswith(":"):
            out.append(None)
            continue
        op, _, rest = s.partition(" ")
        out.append((op, rest.strip(), in_asm))
    return out


def _vregs(text):
    regs = set()
    for m in REG.finditer(text):
        if m.group(3) is not None:
            regs.add(int(m.group(3)))
        else:
            regs.update(range(int(m.group(1)), int(m.group(2)) + 1))
    return regs


def _wait_states(ins):
    return int(ins[1], 0) + 1 if ins[0] == "s_nop" else 1


def test_no_vector_alu_instruction_in_inline_asm(listings):
    for src, lines in listings.items():
        bad = [i for i in _instructions(lines) if i and i[2] and i[0].startswith("v_")]
        assert not bad, f"{src}: VALU instruction in inline asm: {bad[:3]}"


def test_lds_dma_asm_waits_after_its_m0_write(listings):
    n = 0
    for src, lines in listings.items():
        ins = _instructions(lines)
        for k, i in enumerate(ins):
            if not i or not i[2] or not i[0].startswith("global_load_lds"):
                continue
            n += 1
            # walk back to the M0 write of the same asm statement
            ws, j = 0, k - 1
            while j >= 0 and ins[j] and not (ins[j][0].startswith("s_mov") and
                                             ins[j][1].startswith("m0")):
                ws += _wait_states(ins[j])
                j -= 1
            assert j >= 0 and ins[j], f"{src}: LDS DMA without its M0 write"
            assert ws >= 1, f"{src}: LDS DMA issued right after its M0 write"
    assert n > 0


def test_permlane_swaps_are_compiler_placed_with_wait_states(listings):
    """Every swap comes from the builtins, and at least two wait states
    separate it from the last VALU write of either operand in its run."""
    n = 0
    for src, lines in listings.items():
        ins = _instructions(lines)
        for k, i in enumerate(ins):
            if not i or not i[0].startswith("v_permlane") or "swap" not in i[0]:
                continue
            n += 1
            assert not i[2], f"{src}: permlane swap in inline asm"
            ops = _vregs(i[1])
            ws, j = 0, k - 1
            while j >= 0 and ins[j] and ws < 8:
                op, rest, _ = ins[j]
                if op.startswith("v_") and _vregs(rest.split(",")[0]) & ops:
                    assert ws >= 2, f"{src}: {op} then {i[0]} after {ws} wait states"
                    break
                ws += _wait_states(ins[j])
                j -= 1
    assert n > 0


def _functions(lines):
    """{kernel symbol: its lines}, from each function label to its end marker."""
    out, cur = {}, None
    for raw in lines:
        m = re.match(r"^(_Z\w+):", raw)
        if m:
            cur = m.group(1)
            out[cur] = []
            continue
        if cur is not None:
            if raw.startswith(".Lfunc_end"):
                cur = None
                continue
            out[cur].append(raw)
    return out


def test_no_spill_traffic_inside_dma_loops(listings):
    """The LDS DMA is inline assembly, so the compiler does not count it in
    the vector-memory counter it waits on: a spill reload inside a stage loop
    waits with a count that, in hardware, also covers every DMA issued before
    it, and the ring drains to one stage in flight (a build that spilled
    there ran at half speed).  No loop of a kernel that streams through LDS
    DMA may touch scratch memory."""
    n = 0
    for src, lines in listings.items():
        for name, body in _functions(lines).items():
            if not any("global_load_lds" in l for l in body):
                continue
            n += 1
            in_loop, bad = False, []
            for raw in body:
                if re.match(r"^\.LBB\d+_\d+:", raw):
                    in_loop = "Loop" in raw
                    continue
                s = raw.strip().split(";")[0].strip()
                if in_loop and s.startswith(("scratch_", "buffer_store", "buffer_load")):
                    bad.append(s)
            assert not bad, f"{src}: {name} touches scratch inside a loop: {bad[:3]}"
    assert n > 0
