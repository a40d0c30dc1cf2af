"""The LDS fragment reads that the bf16 GEMM and attention kernels issue as
inline assembly are invisible to the compiler's hazard recognizer, so the
generated gfx950 code is checked here instead (CPU only: hipcc emits the
device assembly without a GPU).

An MFMA reads its accumulator input (SrcC) over several passes after it
issues, so a later write of one of those registers needs wait states; the
A and B operands are read at issue.  The check: on every control-flow path,
no inline LDS read writes a register that an MFMA issued within the previous
WINDOW wait states reads as SrcC.  Beside it, as evidence for the A/B rule,
the compiler's own LDS reads in the same files overwrite the A or B operand
of the MFMA issued directly before them (no wait states at all)."""
import os
import re
import subprocess
import tempfile
from collections import defaultdict

import pytest

from paper_2503_03182_amd import build as B

WINDOW = 20
SOURCES = ("gemm_nt.hip", "gemm_nn.hip", "gemm_tn.hip", "attention_fwd.hip", "attention_bwd.hip")
REG = re.compile(r"([va])(?:\[(\d+):(\d+)\]|(\d+))")


def _regs(tok):
    m = REG.fullmatch(tok.strip())
    if not m:
        return set()
    a, b = (int(m.group(4)),) * 2 if m.group(4) is not None else (int(m.group(2)), int(m.group(3)))
    return {(m.group(1), i) for i in range(a, b + 1)}


def _functions(text):
    name, cur = None, None
    for line in text.splitlines():
        m = re.match(r"^([A-Za-z_$][\w.$]*):\s*(;.*)?$", line)
        if m:
            name, cur = m.group(1), []
            continue
        if cur is None:
            continue
        if line.startswith(".Lfunc_end"):
            yield name, cur
            name, cur = None, None
            continue
        cur.append(line)


def _blocks(lines):
    """Basic blocks [(label, [(mnemonic, operands, inline)])]."""
    blocks, inline = [("entry", [])], False
    for line in lines:
        s = line.strip()
        if s.startswith(";;#ASMSTART"):
            inline = True
            continue
        if s.startswith(";;#ASMEND"):
            inline = False
            continue
        if not s or s.startswith(";") or s.startswith("."):
            m = re.match(r"^(\.L\w+):", s)
            if m:
                blocks.append((m.group(1), []))
            continue
        s = s.split(";")[0].strip()
        if not s:
            continue
        parts = s.split(None, 1)
        ops = [o.strip() for o in parts[1].split(",")] if len(parts) > 1 else []
        blocks[-1][1].append((parts[0], ops, inline))
        if parts[0].startswith(("s_branch", "s_cbranch", "s_setpc")) or parts[0] == "s_endpgm":
            blocks.append((None, []))
    return [b for b in blocks if b[0] or b[1]]


def _preds(blocks):
    idx = {b[0]: i for i, b in enumerate(blocks) if b[0]}
    preds = defaultdict(set)
    for i, (_, ins) in enumerate(blocks):
        fall = True
        if ins:
            mn, ops, _ = ins[-1]
            if mn.startswith(("s_branch", "s_setpc")) or mn == "s_endpgm":
                fall = False
            if mn.startswith(("s_branch", "s_cbranch")) and ops and ops[0] in idx:
                preds[idx[ops[0]]].add(i)
        if fall and i + 1 < len(blocks):
            preds[i + 1].add(i)
    return preds


def _wait_states(instr):
    return int(instr[1][0], 0) + 1 if instr[0] == "s_nop" else 1


def scan(text, window=WINDOW):
    """-> list of (kernel, inline, operand, wait states, destination) for every LDS read
    whose destination overlaps operand A, B or C of an MFMA issued fewer than
    `window` wait states before it on some path."""
    hits = []
    for name, lines in _functions(text):
        blocks = _blocks(lines)
        preds = _preds(blocks)
        for bi, (_, ins) in enumerate(blocks):
            for ii, (mn, ops, inline) in enumerate(ins):
                if not mn.startswith("ds_read"):
                    continue
                dst = _regs(ops[0])
                stack, seen = [(bi, ii - 1, 0)], set()
                while stack:
                    b, j, d = stack.pop()
                    if (b, j, d) in seen:
                        continue
                    seen.add((b, j, d))
                    if j < 0:
                        stack += [(p, len(blocks[p][1]) - 1, d) for p in preds[b]]
                        continue
                    instr = blocks[b][1][j]
                    if instr[0].startswith("v_mfma"):
                        o = instr[1]
                        for k, tok in (("A", o[1]), ("B", o[2]), ("C", o[3])):
                            if dst & _regs(tok):
                                hits.append((name, inline, k, d, ops[0]))
                    nd = d + _wait_states(instr)
                    if nd < window:
                        stack.append((b, j - 1, nd))
    return hits


@pytest.fixture(scope="module")
def assembly():
    out = {}
    with tempfile.TemporaryDirectory() as tmp:
        procs = []
        for src in SOURCES:
            dst = os.path.join(tmp, src + ".s")
            cmd = [B.hipcc(), "-x", "hip", *B.COMMON, *B.DEVICE_FLAGS, "--cuda-device-only", "-S",
                   os.path.join(B.CSRC, src), "-o", dst]
            procs.append((src, dst, subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.PIPE)))
        for src, dst, p in procs:
            _, err = p.communicate()
            assert p.returncode == 0, (src, err.decode()[-2000:])
            out[src] = open(dst).read()
    return out


def test_scanner_finds_planted_overlaps():
    text = "\n".join([
        "k:",
        "\tv_mfma_f32_32x32x16_bf16 v[0:15], v[16:19], v[20:23], v[0:15]",
        "\ts_nop 3",
        "\t;;#ASMSTART",
        "\tds_read_b128 v[12:15], v30 offset:0",
        "\t;;#ASMEND",
        "\tds_read_b128 v[16:19], v31 offset:0",
        ".LBB0_1:",
        "\tv_mfma_f32_32x32x16_bf16 v[32:47], v[48:51], v[52:55], v[32:47]",
        "\ts_cbranch_scc1 .LBB0_1",
        "\t;;#ASMSTART",
        "\tds_read_b64_tr_b16 v[46:47], v30 offset:0",
        "\t;;#ASMEND",
        "\ts_nop 15",
        "\ts_nop 15",
        "\tds_read_b128 v[32:35], v30 offset:0",
        ".Lfunc_end0:",
    ])
    hits = {(h[4], h[1], h[2], h[3]) for h in scan(text)}
    assert ("v[12:15]", True, "C", 4) in hits     # after s_nop 3: 4 wait states
    assert ("v[16:19]", False, "A", 5) in hits
    assert ("v[46:47]", True, "C", 1) in hits     # through the loop's exit edge
    assert ("v[46:47]", True, "C", 3) in hits     # and once more round the loop
    assert not any(h[0] == "v[32:35]" for h in hits)   # 32 wait states back


def test_inline_lds_reads_never_overwrite_mfma_accumulator_inputs(assembly):
    n_inline_reads = 0
    for src, text in assembly.items():
        n_inline_reads += len(re.findall(r";;#ASMSTART\s*\n\s*ds_read", text))
        bad = [h for h in scan(text) if h[1] and h[2] == "C"]
        assert not bad, (src, bad[:5])
    assert n_inline_reads > 1000


def test_compiler_reads_overwrite_mfma_ab_operands_without_wait_states(assembly):
    """The toolchain's own code: a compiler-issued LDS read writes the A or B
    operand registers of the MFMA directly before it, which the compiler's
    hazard model allows only because A and B are read at issue."""
    found = []
    for src, text in assembly.items():
        found += [h for h in scan(text, window=1) if not h[1] and h[2] in "AB"]
    assert found
