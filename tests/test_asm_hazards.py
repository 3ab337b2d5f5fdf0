"""Inline-asm hazards of the HIP kernels, checked on the CPU.

The kernels issue their global->LDS copies from inline asm that sets M0 with a
scalar add, which also writes SCC (the scalar carry / condition bit). The
compiler only keeps a value in SCC across an asm statement that does not
declare the clobber, so two checks guard against a copy landing between an
SCC producer and its consumer (for instance between the two halves of a
64-bit scalar pointer add, which then loses its carry and points 4 GiB off
whenever the low half wraps):

* source: every asm template that runs a scalar ALU instruction declares "scc";
* assembly: in the device code of every build part, no instruction that reads
  SCC takes it from before an asm block that writes SCC.

The query rows are loaded by asm straight into AGPRs, and a later asm waits
for them (vmcnt). The compiler sees the registers as written when the load
statement ends, so the assembly check also makes sure that no instruction
touches them before that wait.
"""
import os
import re
import shutil
import subprocess

import pytest

from paper_2608_26523_amd import build as BLD

# scalar ALU instructions that write SCC (the ones the kernels' asm or the
# compiler's pointer and index arithmetic use)
SCC_WRITE = re.compile(
    r"^s_(add|sub|addc|subb|addk|and|or|xor|andn2|orn2|nand|nor|xnor|not|lshl|lshr|ashr|bfe|"
    r"cmp|cmpk|min|max|abs|absdiff|bcnt|bitcmp|quadmask|wqm)[a-z0-9_]*$")
SCC_READ = re.compile(r"^s_(addc_u32|subb_u32|cselect_b32|cselect_b64|cmov_b32|cmov_b64|cmovk_i32|"
                      r"cbranch_scc0|cbranch_scc1)$")


def _asm_statements(src: str):
    """(template, clobbers) of every asm statement of the source."""
    out = []
    for m in re.finditer(r"\basm\s*(volatile\s*)?\(", src):
        i, depth = m.end(), 1
        while depth:
            depth += {"(": 1, ")": -1}.get(src[i], 0)
            i += 1
        body = src[m.end():i - 1]
        parts = body.split(":")
        template = "".join(re.findall(r'"((?:[^"\\]|\\.)*)"', parts[0]))
        clobbers = re.findall(r'"([^"]*)"', parts[3]) if len(parts) > 3 else []
        out.append((template, clobbers))
    return out


def test_scalar_alu_asm_declares_scc():
    src = open(BLD.SRC).read()
    stmts = _asm_statements(src)
    assert len(stmts) >= 10
    writers = 0
    for template, clobbers in stmts:
        ops = [ln.split()[0] for ln in template.replace("\\n", "\n").replace("\\t", "").splitlines()
               if ln.strip()]
        if any(SCC_WRITE.match(op) for op in ops):
            writers += 1
            assert "scc" in clobbers, "asm writes SCC without declaring it: %r" % template
    assert writers >= 1  # the LDS copy


def _scan(asm_text: str):
    """Instructions reading an SCC value that an SCC-writing asm block overwrote."""
    hits = []
    live = False      # an SCC value produced by compiled code may be in use
    clobbered = False
    in_asm = asm_writes = False
    for n, line in enumerate(asm_text.splitlines(), 1):
        if ";;#ASMSTART" in line:
            in_asm, asm_writes = True, False
            continue
        if ";;#ASMEND" in line:
            in_asm = False
            if asm_writes and live:
                clobbered = True
            continue
        code = line.split(";")[0].strip()
        if not code:
            continue
        if code.endswith(":"):          # block label: values do not flow in from here
            live = clobbered = False
            continue
        op = code.split()[0]
        if in_asm:
            asm_writes = asm_writes or bool(SCC_WRITE.match(op))
            continue
        if SCC_READ.match(op) and clobbered:
            hits.append((n, code))
        if SCC_WRITE.match(op):
            live, clobbered = True, False
    return hits


def _agprs(text: str):
    regs = set()
    for m in re.finditer(r"a\[(\d+):(\d+)\]", text):
        regs.update(range(int(m.group(1)), int(m.group(2)) + 1))
    for m in re.finditer(r"\ba(\d+)\b", text):
        regs.add(int(m.group(1)))
    return regs


def _scan_async_agpr(asm_text: str):
    """(loads, instructions touching an AGPR of an asm global load before its vmcnt wait)."""
    hits, pending, loads = [], set(), 0
    in_asm, block = False, []
    for n, line in enumerate(asm_text.splitlines(), 1):
        if ";;#ASMSTART" in line:
            in_asm, block = True, []
            continue
        if ";;#ASMEND" in line:
            in_asm = False
            for ins in block:
                if ins.startswith("global_load") and " a" in ins.split(",")[0]:
                    loads += 1
                    pending |= _agprs(ins.split(",")[0])
                elif ins.startswith("s_waitcnt") and "vmcnt(0)" in ins:
                    pending = set()
            continue
        code = line.split(";")[0].strip()
        if in_asm:
            if code:
                block.append(code)
            continue
        if not code or code.endswith(":"):
            continue
        if code.startswith("s_waitcnt") and "vmcnt(0)" in code:
            pending = set()
        elif pending and _agprs(code) & pending:
            hits.append((n, code))
    return loads, hits


def test_scan_finds_a_planted_hazard():
    planted = "\n".join([
        "\ts_add_u32 s4, s4, s6",
        "\t;;#ASMSTART",
        "\ts_add_u32 m0, s10, 0x1000",
        "\t;;#ASMEND",
        "\ts_addc_u32 s5, s5, s7",
    ])
    assert len(_scan(planted)) == 1
    fixed = planted.replace("\ts_addc_u32", "\ts_add_u32 s8, s8, s9\n\ts_addc_u32")
    assert _scan(fixed) == []
    early = "\n".join([
        "\t;;#ASMSTART",
        "\tglobal_load_dwordx4 a[4:7], v2, off",
        "\t;;#ASMEND",
        "\tv_accvgpr_read_b32 v9, a5",
        "\t;;#ASMSTART",
        "\ts_waitcnt vmcnt(0)",
        "\t;;#ASMEND",
        "\tv_accvgpr_read_b32 v10, a6",
    ])
    loads, hits = _scan_async_agpr(early)
    assert loads == 1 and [h[1] for h in hits] == ["v_accvgpr_read_b32 v9, a5"]


@pytest.mark.skipif(not os.path.exists(BLD.hipcc()), reason="hipcc not installed")
def test_device_code_asm_hazards(tmp_path):
    base = [BLD.hipcc()] + [f for f in BLD.HIPCC_FLAGS if f not in ("-shared", "-Wall")] + ["-I", BLD.INCLUDE]
    procs = []
    for part in BLD.PARTS:
        out = str(tmp_path / ("part%d.s" % part))
        cmd = base + ["--cuda-device-only", "-S", "-DVPP_PART=%d" % part, "-o", out, BLD.SRC]
        procs.append((part, out, subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT,
                                                   text=True)))
    for part, out, pr in procs:
        log = pr.communicate(timeout=600)[0]
        assert pr.returncode == 0, log[-2000:]
        text = open(out).read()
        assert "buffer_load_dwordx4" in text and ";;#ASMSTART" in text
        hits = _scan(text)
        assert hits == [], "part %d: SCC read after an SCC-writing asm block: %s" % (part, hits[:5])
        loads, early = _scan_async_agpr(text)
        assert loads > 0, "part %d: no asm query loads found" % part
        assert early == [], "part %d: query AGPRs used before their load completed: %s" % (part, early[:5])
    shutil.rmtree(tmp_path, ignore_errors=True)
