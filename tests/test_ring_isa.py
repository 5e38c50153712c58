"""The select kernel's prefetch ring, checked in the gfx950 assembly the
compiler produces for it (CPU only: hipcc cross-compiles).

The ring loads key tiles with inline-assembly loads and waits for them with
explicit vmcnt counts.  The compiler believes such a load writes its
registers at once, so any instruction it places between the load and the
wait that covers it and that reads those registers (a copy at a loop
back-edge, a dynamically indexed move) would read data that has not landed.
This test compiles select.hip to assembly and walks forward from every ring
load, in program order, until a wait that covers it (loads complete in
issue order, so vmcnt(n) covers a load once at least n vector-memory
instructions were issued after it) and fails on any read of its registers
before that point.  Walking in program order across branches is
conservative for straight-line code and catches the back-edge copies,
which sit at the end of the loop body.
"""
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2604_03815_amd", "csrc")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

RING_LOAD = re.compile(r"global_load_dword(?:x4)? (?:v\[(\d+):(\d+)\]|v(\d+)), v\d+, s\[\d+:\d+\]")
WAIT = re.compile(r"s_waitcnt vmcnt\((\d+)\)")
VMEM = ("global_load", "global_store", "global_atomic", "buffer_load", "buffer_store", "flat_load",
        "flat_store")


def _regs(text):
    out = set()
    for m in re.finditer(r"v\[(\d+):(\d+)\]", text):
        out |= set(range(int(m.group(1)), int(m.group(2)) + 1))
    for m in re.finditer(r"\bv(\d+)\b", text):
        out.add(int(m.group(1)))
    return out


LABEL = re.compile(r"^(\.LBB\w+|\.Ltmp\w+):")
BRANCH = re.compile(r"^s_(c?branch)\w*\s+(\.\w+)")


def early_reads(body):
    """(load, offending instruction) pairs of one kernel's assembly lines.

    From every ring load, every control-flow path is followed (fall-through,
    and the targets of s_branch and s_cbranch_*) up to a wait that covers the
    load; a path that reads one of the load's registers first is reported.
    Registers that a path overwrites drop out of that path's live set."""
    labels = {}
    for i, line in enumerate(body):
        m = LABEL.match(line)
        if m:
            labels[m.group(1)] = i
    found = []
    for i, line in enumerate(body):
        m = RING_LOAD.match(line)
        if not m:
            continue
        live0 = frozenset(range(int(m.group(1)), int(m.group(2)) + 1)) if m.group(1) else frozenset({int(m.group(3))})
        stack = [(i + 1, 0, live0)]
        seen = set()
        hit = None
        while stack and hit is None:
            pos, issued_after, live = stack.pop()
            while pos < len(body):
                state = (pos, min(issued_after, 64), live)
                if state in seen:
                    break
                seen.add(state)
                x = body[pos]
                if not x or x.startswith((";", ".")):
                    pos += 1
                    continue
                w = WAIT.match(x)
                if w and int(w.group(1)) <= issued_after:
                    break
                op = x.split()[0]
                if op.startswith(VMEM):
                    issued_after += 1
                if op.startswith("s_"):
                    br = BRANCH.match(x)
                    if br and br.group(2) in labels:
                        stack.append((labels[br.group(2)] + 1, issued_after, live))
                        if br.group(1) == "branch":
                            break          # unconditional: no fall-through
                    elif op in ("s_endpgm", "s_setpc_b64"):
                        break
                    pos += 1
                    continue
                fields = x.split(None, 1)
                if len(fields) < 2:
                    pos += 1
                    continue
                operands = fields[1].split(",")
                stores = op.startswith(("global_store", "buffer_store", "flat_store", "ds_write"))
                sources = fields[1] if stores else ",".join(operands[1:])
                if _regs(sources) & live:
                    hit = (line, x)
                    break
                if not stores and not op.startswith("v_cmp"):
                    live = live - _regs(operands[0])
                    if not live:
                        break
                pos += 1
        if hit is not None:
            found.append(hit)
    return found


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="no hipcc")
def test_no_ring_register_is_read_before_its_wait(tmp_path):
    out = tmp_path / "select.s"
    cmd = [HIPCC, "-O3", "-std=c++17", "--offload-arch=gfx950", "--cuda-device-only", "-S",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", "-fno-honor-nans",
           "-mllvm", "-amdgpu-mfma-vgpr-form=1", "-I", os.path.join(ROOT, "include"), "-I", CSRC,
           os.path.join(CSRC, "select.hip"), "-o", str(out)]
    subprocess.run(cmd, check=True, stdout=subprocess.DEVNULL, stderr=subprocess.DEVNULL, timeout=600)
    text = out.read_text()
    kernels = re.split(r"\n(?=_ZN4kmip\S*select_kernel\S*:)", text)[1:]
    assert kernels, "no select kernel in the assembly"
    problems = {}
    for k in kernels:
        name = k.split(":")[0]
        body = [l.strip() for l in k[:k.find(".Lfunc_end")].splitlines()]
        assert any(RING_LOAD.match(l) for l in body), name
        bad = early_reads(body)
        if bad:
            problems[name] = bad[:3]
    assert not problems, problems


def test_checker_flags_a_copy_before_the_wait():
    # the pattern the compiler produced once for a prefetched index register
    body = ["global_load_dword v168, v127, s[0:1]",
            "v_mov_b32_e32 v175, v168",
            "s_waitcnt vmcnt(0)"]
    assert early_reads(body)
    ok = ["global_load_dwordx4 v[2:5], v121, s[0:1] offset:0",
          "global_load_dwordx4 v[6:9], v121, s[2:3] offset:0",
          "s_waitcnt vmcnt(1)",
          "v_mfma_f32_32x32x16_bf16 v[10:25], v[2:5], v[30:33], 0",
          "v_mov_b32_e32 v40, v6"]
    # v[2:5] is covered by vmcnt(1) (one load issued after it); v[6:9] is not
    assert early_reads(ok) == [(ok[1], ok[4])]


def test_checker_follows_branches():
    # a read of the ring register at a branch target is caught; one that only
    # follows an unconditional branch in the layout is not on any path
    body = ["global_load_dwordx4 v[2:5], v121, s[0:1] offset:0",
            "s_cbranch_scc0 .LBB0_2",
            "s_waitcnt vmcnt(0)",
            "s_branch .LBB0_3",
            "v_mov_b32_e32 v40, v2",
            ".LBB0_2:",
            "v_mov_b32_e32 v41, v3",
            ".LBB0_3:",
            "s_endpgm"]
    assert early_reads(body) == [(body[0], body[6])]
    body[1] = "s_cbranch_scc0 .LBB0_3"
    assert early_reads(body) == []
    # a loop back-edge that reaches the read before the wait
    loop = [".LBB0_1:",
            "v_mov_b32_e32 v41, v3",
            "s_waitcnt vmcnt(0)",
            "global_load_dwordx4 v[2:5], v121, s[0:1] offset:0",
            "s_cbranch_scc1 .LBB0_1",
            "s_waitcnt vmcnt(0)",
            "s_endpgm"]
    assert early_reads(loop) == [(loop[3], loop[1])]
