"""Wait states around the fused backward kernel's hand-placed MFMAs (CPU only).

k_bwd_fused accumulates every group's sums with MFMAs written as inline
assembly (accumulators in AGPRs).  The compiler's hazard recognizer does not
see inside those statements, so the kernel waits out the MFMA latency itself
(agpr_settle at the end of every tile) before anything else may touch an
accumulator.  This test compiles the kernel file to gfx950 assembly with the
library's flags and checks, over the control-flow graph of each k_bwd_fused
instance, that no instruction other than those MFMAs reads or writes an AGPR
that such an MFMA has written since the last settle; a copy of the assembly
with the settle removed must fail the same check.
"""
import os
import re
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SETTLE = "s_nop 7 ; s_nop 7 ; s_nop 7"


def _blocks(lines, start, end):
    """Basic blocks of one function: (label, [(kind, text)]) and successors."""
    blocks, cur, in_asm, asm = [], {"label": None, "ins": []}, False, []
    for raw in lines[start + 1:end]:
        s = raw.strip()
        m = re.match(r"^(\.LBB\S+):", raw)
        if m:
            blocks.append(cur)
            cur = {"label": m.group(1), "ins": []}
            continue
        if s.startswith(";;#ASMSTART"):
            in_asm, asm = True, []
            continue
        if s.startswith(";;#ASMEND"):
            in_asm = False
            cur["ins"].append(("asm", " ; ".join(asm)))
            continue
        if in_asm:
            asm.append(s)
            continue
        if not s or s.startswith(";") or s.startswith("."):
            continue
        text = s.split(";")[0].strip()
        cur["ins"].append(("ins", text))
        op = text.split()[0]
        if op.startswith("s_cbranch") or op in ("s_branch", "s_endpgm") or op.startswith("s_setpc"):
            blocks.append(cur)
            cur = {"label": None, "ins": []}
    blocks.append(cur)
    blocks = [b for b in blocks if b["ins"] or b["label"]]
    index = {b["label"]: k for k, b in enumerate(blocks) if b["label"]}
    succ = []
    for k, b in enumerate(blocks):
        last = b["ins"][-1][1] if b["ins"] else ""
        op = last.split()[0] if last else ""
        s = [index[last.split()[1]]] if (op.startswith("s_cbranch") or op == "s_branch") else []
        if op not in ("s_branch", "s_endpgm") and k + 1 < len(blocks):
            s.append(k + 1)
        succ.append(s)
    return blocks, succ


def _agprs(text):
    regs = set()
    for m in re.finditer(r"\ba\[(\d+):(\d+)\]", text):
        regs |= set(range(int(m.group(1)), int(m.group(2)) + 1))
    for m in re.finditer(r"\ba(\d+)\b", text):
        regs.add(int(m.group(1)))
    return regs


def _run(block, pending, bad=None):
    pending = set(pending)
    for kind, text in block["ins"]:
        if kind == "asm":
            m = re.search(r"v_mfma\S*\s+a\[(\d+):(\d+)\]", text)
            if m:
                pending |= set(range(int(m.group(1)), int(m.group(2)) + 1))
            elif text == SETTLE:
                pending = set()
            continue
        if bad is not None and _agprs(text) & pending:
            bad.append(text)
    return pending


def hazards(asm_text, kernel):
    """{function: (asm MFMAs, violating instructions)} for every instance of `kernel`."""
    lines = asm_text.split("\n")
    out = {}
    for start in [i for i, l in enumerate(lines) if re.match(r"^_Z\S*" + kernel + r"\S*:", l)]:
        end = next(i for i in range(start, len(lines)) if lines[i].startswith(".Lfunc_end"))
        blocks, succ = _blocks(lines, start, end)
        entry = [set() for _ in blocks]
        changed = True
        while changed:  # pending AGPRs at each block entry: union over the predecessors
            changed = False
            for k, b in enumerate(blocks):
                after = _run(b, entry[k])
                for s in succ[k]:
                    if not after <= entry[s]:
                        entry[s] |= after
                        changed = True
        bad = []
        for k, b in enumerate(blocks):
            _run(b, entry[k], bad)
        n_mfma = sum(1 for b in blocks for kind, t in b["ins"] if kind == "asm" and "v_mfma" in t)
        out[lines[start].split(":")[0]] = (n_mfma, bad)
    return out


@pytest.fixture(scope="module")
def backward_asm(tmp_path_factory):
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(hipcc):
        pytest.skip("hipcc not found")
    sys.path.insert(0, os.path.join(ROOT, "paper_2306_01926_amd"))
    from build import DEVICE_FLAGS

    out = str(tmp_path_factory.mktemp("asm") / "ga_backward.s")
    src = os.path.join(ROOT, "paper_2306_01926_amd", "csrc", "ga_backward.hip")
    r = subprocess.run([hipcc, *DEVICE_FLAGS, "--cuda-device-only", "-S", "-o", out, src],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-3000:]
    return open(out).read()


def test_fused_backward_accumulators_settle_before_use(backward_asm):
    found = hazards(backward_asm, "k_bwd_fused")
    assert len(found) == 4, sorted(found)  # NB = 1 .. 4
    for name, (n_mfma, bad) in found.items():
        assert n_mfma > 0, name
        assert not bad, (name, bad[:5])


def test_hazard_check_sees_a_missing_settle(backward_asm):
    planted = backward_asm.replace("\ts_nop 7\n\ts_nop 7\n\ts_nop 7", "\ts_nop 6\n\ts_nop 7\n\ts_nop 7")
    assert planted != backward_asm
    found = hazards(planted, "k_bwd_fused")
    assert found and all(bad for _, bad in found.values())
