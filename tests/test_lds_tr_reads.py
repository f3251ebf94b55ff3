"""The transposing LDS reads that the GEMM issues as inline assembly are
outside the compiler's wait and hazard tracking: the code waits for them
itself (lgkmcnt(0)) and pins their results behind that wait.  This test
compiles csrc/gemm.hip for gfx950 to assembly and checks, by a dataflow
pass over each kernel's control-flow graph, that on every path from such a
read to the next wait covering it (an s_waitcnt with lgkmcnt(0)) no
instruction reads or writes the read's destination registers, and that no
read uses an address register still being written by an earlier read.  A
planted violation (an instruction touching a destination register right
after a read) must be reported.  CPU only: needs hipcc, no GPU."""
import os
import re
import shutil
import subprocess

import pytest

import paper_2202_11836_amd.build as B

SRC = os.path.join(B.CSRC, "gemm.hip")


def _vregs(text):
    out = set()
    for m in re.finditer(r"\bv\[(\d+):(\d+)\]", text):
        out |= set(range(int(m.group(1)), int(m.group(2)) + 1))
    for m in re.finditer(r"\bv(\d+)\b", text):
        out.add(int(m.group(1)))
    return out


def check_asm(text):
    """Problems found in gfx9 assembly text, and the number of hand-issued
    transposing reads seen."""
    problems, nreads = [], 0
    funcs, cur = [], None
    for ln, line in enumerate(text.split("\n"), 1):
        s = line.strip()
        m = re.match(r"^(_Z\w+):", s)
        if m:
            cur = (m.group(1), [])
            funcs.append(cur)
            continue
        if cur is not None:
            if s.startswith(".Lfunc_end"):
                cur = None
            else:
                cur[1].append((ln, s))
    for name, body in funcs:
        items, inasm = [], False
        for ln, s in body:
            if s.startswith(";;#ASMSTART"):
                inasm = True
            elif s.startswith(";;#ASMEND"):
                inasm = False
            elif not s or s.startswith(";"):
                continue
            elif re.match(r"^(\.?L\w+):", s):
                items.append((ln, "label", s.split(":")[0], False))
            elif not s.startswith("."):
                items.append((ln, "ins", s, inasm))
        blocks, cb = [], []
        for it in items:
            if it[1] == "label":
                if cb:
                    blocks.append(cb)
                cb = [it]
                continue
            cb.append(it)
            op = it[2].split()[0]
            if op.startswith("s_cbranch") or op in ("s_branch", "s_endpgm", "s_setpc_b64"):
                blocks.append(cb)
                cb = []
        if cb:
            blocks.append(cb)
        at = {b[0][2]: i for i, b in enumerate(blocks) if b[0][1] == "label"}
        succ = []
        for i, b in enumerate(blocks):
            last, nxt = b[-1], []
            op = last[2].split()[0] if last[1] == "ins" else ""
            if op.startswith("s_cbranch"):
                nxt = [at[last[2].split()[1]], i + 1]
            elif op == "s_branch":
                nxt = [at[last[2].split()[1]]]
            elif op not in ("s_endpgm", "s_setpc_b64"):
                nxt = [i + 1]
            succ.append([j for j in nxt if j < len(blocks)])

        def run(block, pend, report):
            pend = dict(pend)
            for ln, kind, s, inasm in block:
                if kind != "ins":
                    continue
                op = s.split()[0]
                rest = s[len(op):]
                if op == "ds_read_b64_tr_b16" and inasm:
                    dst, addr = rest.split(",")[0], rest.split(",", 1)[1]
                    if report is not None and _vregs(addr) & set(pend):
                        report.append(f"{name}:{ln}: read address still being written")
                    for r in _vregs(dst):
                        pend[r] = ln
                elif op == "s_waitcnt":
                    if "lgkmcnt(0)" in rest:
                        pend = {}
                else:
                    hit = _vregs(rest) & set(pend)
                    if hit and report is not None:
                        report.append(f"{name}:{ln}: '{s[:60]}' touches v{min(hit)} "
                                      f"(read at line {pend[min(hit)]})")
            return pend

        state = [None] * len(blocks)
        if blocks:
            state[0] = {}
        work = [0] if blocks else []
        while work:
            i = work.pop()
            out = run(blocks[i], state[i], None)
            for j in succ[i]:
                new = dict(state[j] or {})
                changed = state[j] is None
                for r, l in out.items():
                    if r not in new:
                        new[r] = l
                        changed = True
                if changed:
                    state[j] = new
                    work.append(j)
        for i, b in enumerate(blocks):
            if state[i] is not None:
                run(b, state[i], problems)
        nreads += sum(1 for b in blocks for it in b
                      if it[1] == "ins" and it[3] and it[2].startswith("ds_read_b64_tr_b16"))
    return problems, nreads


@pytest.fixture(scope="module")
def gemm_asm(tmp_path_factory):
    if shutil.which(B.HIPCC) is None and not os.path.exists(B.HIPCC):
        pytest.skip("hipcc not found")
    out = tmp_path_factory.mktemp("asm") / "gemm.s"
    flags = [f for f in B.COMMON_FLAGS if f != "-fPIC"]
    r = subprocess.run([B.HIPCC] + flags + ["--cuda-device-only", "-S", SRC, "-o", str(out)],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    return out.read_text()


def test_hand_issued_transposing_reads_are_waited_for(gemm_asm):
    problems, nreads = check_asm(gemm_asm)
    assert nreads > 0, "no hand-issued transposing reads found"
    assert not problems, "\n".join(problems[:20])


def test_checker_reports_a_planted_violation(gemm_asm):
    m = re.search(r";;#ASMSTART\n\s*ds_read_b64_tr_b16 v\[(\d+):\d+\].*\n\s*;;#ASMEND\n", gemm_asm)
    assert m
    planted = gemm_asm[:m.end()] + f"\tv_mov_b32_e32 v{m.group(1)}, 0\n" + gemm_asm[m.end():]
    problems, _ = check_asm(planted)
    assert any("touches" in p for p in problems)
