"""Wait states around the MFMAs the kernels write as inline assembly (CPU).

The compiler inserts the wait states the matrix cores need around its own
MFMAs, but treats an MFMA inside an `asm` statement as an opaque instruction.
The kv pass issues its S/dP products that way (vector-register accumulators),
so this test compiles the kernels to gfx950 assembly with the library's flags
and checks, on every path of the control flow, the rules the hand-written
products rely on:

* an operand (A, B, or C) of the MFMA is not written by a vector ALU
  instruction in the 2 wait states before it;
* no instruction other than a product chained on the same registers reads or
  writes the MFMA's result, or writes its C operand, in the 19 wait states
  after it (the longest 32x32 product).

A wait state is one issued instruction, or N + 1 for `s_nop N`.
"""
import os
import re
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, os.path.join(ROOT, "paper_2607_21624_amd"))
import build as fbl_build  # noqa: E402

BEFORE = 2
AFTER = 19
SOURCES = ["attn_bwd_kv.hip"]


def _regs(tok):
    tok = tok.strip().lstrip("-")
    m = re.match(r"v\[(\d+):(\d+)\]$", tok)
    if m:
        return set(range(int(m.group(1)), int(m.group(2)) + 1))
    m = re.match(r"v(\d+)$", tok)
    return {int(m.group(1))} if m else set()


class Fn:
    """One kernel: instructions (text), labels and control-flow edges."""

    def __init__(self, lines):
        self.ins = []     # (mnemonic, operands list, raw, in_asm)
        self.label_at = {}
        in_asm = False
        for l in lines:
            s = l.strip()
            if s.startswith(";;#ASMSTART"):
                in_asm = True
                continue
            if s.startswith(";;#ASMEND"):
                in_asm = False
                continue
            m = re.match(r"^(\.LBB\w+):", s)
            if m:
                self.label_at[m.group(1)] = len(self.ins)
                continue
            if not s or s.startswith(";") or s.startswith("."):
                continue
            s = s.split(";")[0].strip()
            parts = s.split(None, 1)
            ops = [o.strip() for o in parts[1].split(",")] if len(parts) > 1 else []
            self.ins.append((parts[0], ops, s, in_asm))
        self.preds = [[] for _ in self.ins]
        self.succs = [[] for _ in self.ins]
        for i, (mn, ops, _, _) in enumerate(self.ins):
            tgt = self.label_at.get(ops[0]) if mn.startswith(("s_branch", "s_cbranch")) and ops else None
            if tgt is not None:
                self.succs[i].append(tgt)
            if mn not in ("s_branch", "s_endpgm", "s_setpc_b64") and i + 1 < len(self.ins):
                self.succs[i].append(i + 1)
            for j in self.succs[i]:
                self.preds[j].append(i)

    @staticmethod
    def weight(mn, ops):
        if mn == "s_nop":
            return int(ops[0], 0) + 1
        return 1

    def walk(self, start, budget, step):
        """Every instruction reachable from `start` (exclusive) within `budget`
        wait states, following successors (step='f') or predecessors (step='b')."""
        seen = set()
        todo = [(start, budget)]
        while todo:
            i, left = todo.pop()
            for j in (self.succs[i] if step == "f" else self.preds[i]):
                if (j, left) in seen:
                    continue
                seen.add((j, left))
                yield j
                w = self.weight(*self.ins[j][:2])
                if left - w > 0:
                    todo.append((j, left - w))


def _asm_for(src, tmp_path):
    out = tmp_path / (os.path.splitext(src)[0] + ".s")
    cmd = [fbl_build.HIPCC, *fbl_build.FLAGS, "-S", "--offload-device-only", "-o", str(out),
           os.path.join(fbl_build.CSRC, src)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        pytest.fail(r.stdout + r.stderr)
    return out.read_text().split("\n")


def _functions(lines):
    fns, cur, name = {}, None, None
    for l in lines:
        m = re.match(r"^(_Z\w+):", l)
        if m:
            name, cur = m.group(1), []
            continue
        if cur is not None:
            cur.append(l)
            if "s_endpgm" in l:
                fns[name] = Fn(cur)
                cur = None
    return fns


def _is_valu_write(ins, regs):
    mn, ops, _, _ = ins
    return mn.startswith("v_") and "mfma" not in mn and ops and bool(_regs(ops[0]) & regs)


def _problems(fns):
    """(inline-assembly MFMAs checked, hazards found) over the kernels `fns`."""
    checked = 0
    problems = []
    for name, fn in fns.items():
        for i, (mn, ops, raw, in_asm) in enumerate(fn.ins):
            if not (in_asm and mn.startswith("v_mfma")):
                continue
            checked += 1
            dst, a, b, c = (_regs(o) for o in ops[:4])
            for j in fn.walk(i, BEFORE, "b"):
                if _is_valu_write(fn.ins[j], a | b | c):
                    problems.append(f"{name}: '{fn.ins[j][2]}' writes an operand of '{raw}' too late")
            for j in fn.walk(i, AFTER, "f"):
                mn2, ops2, raw2, _ = fn.ins[j]
                if mn2.startswith("v_mfma"):
                    # a product chained on the same accumulator (C = D of this one) may follow at once
                    if len(ops2) > 3 and _regs(ops2[0]) == dst and _regs(ops2[3]) == dst:
                        continue
                    used = set().union(*(_regs(o) for o in ops2[:4]))
                else:
                    used = set().union(*(_regs(o) for o in ops2))
                if used & dst or (not mn2.startswith("v_mfma") and ops2 and _regs(ops2[0]) & c):
                    problems.append(f"{name}: '{raw2}' touches the result or C operand of '{raw}' too early")
    return checked, sorted(set(problems))


def _snippet(body):
    return _functions(["_Zk:"] + [l.strip() for l in body.strip().split("\n")] + ["s_endpgm"])


def test_checker_flags_planted_hazards():
    """The rules themselves, on hand-made assembly: a vector write just
    before an operand, a read of the result just after, and a loop whose
    back edge brings a write too close; the same code with enough wait
    states passes."""
    mfma = ";;#ASMSTART\nv_mfma_f32_32x32x16_bf16 v[0:15], v[16:19], v[20:23], v[0:15]\n;;#ASMEND"
    n, p = _problems(_snippet("v_mov_b32 v17, 0\n" + mfma + "\nv_add_f32_e32 v30, v3, v4"))
    assert n == 1 and len(p) == 2
    n, p = _problems(_snippet("v_mov_b32 v21, 0\ns_nop 1\n" + mfma + "\ns_nop 7\ns_nop 7\ns_nop 3\n"
                              "v_add_f32_e32 v30, v3, v4"))
    assert n == 1 and p == []
    # the C operand written by a vector instruction at the end of a loop, one wait state before the
    # product at its top
    loop = ".LBB0_1:\n" + mfma + "\ns_nop 7\ns_nop 7\ns_nop 7\nv_mov_b32 v5, 0\ns_cbranch_scc1 .LBB0_1"
    n, p = _problems(_snippet(loop))
    assert n == 1 and any("writes an operand" in x for x in p)


@pytest.mark.skipif(not os.path.exists(fbl_build.HIPCC), reason="hipcc not installed")
@pytest.mark.parametrize("src", SOURCES)
def test_inline_mfma_wait_states(src, tmp_path):
    checked, problems = _problems(_functions(_asm_for(src, tmp_path)))
    assert checked > 0, "no inline-assembly MFMA found: the test no longer covers the kv pass"
    assert not problems, "\n".join(problems[:20])
