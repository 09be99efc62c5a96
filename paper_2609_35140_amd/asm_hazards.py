"""Hazard check for the inline assembly in the kernels (build-time check).

The compiler inserts the wait states that gfx950 requires between dependent
instructions only where it generated both of them; an instruction written as
inline asm is opaque to it, so a dependency ending at an asm operand gets no
wait states.  This module compiles kernel sources to gfx950 assembly and
walks back from every instruction that came from inline asm (between the
compiler's ``;;#ASMSTART`` / ``;;#ASMEND`` markers), through fall-through
and branch predecessors, looking for the producers of the registers it reads:

* a transcendental VALU result (``v_exp_f32`` and the like) read by a
  non-transcendental VALU instruction: 1 wait state;
* an SGPR written by a VALU instruction (``v_readfirstlane``, a compare
  into an SGPR pair, ...) read by a vector-memory instruction: 5 wait states;
* a VGPR written by a matrix (MFMA) instruction read by a VALU instruction:
  up to 19 wait states for the longest products (taken for every MFMA).

Every instruction in between counts one wait state (``s_nop n`` counts n+1).

    python -m paper_2609_35140_amd.asm_hazards            # check the kernels
"""
from __future__ import annotations

import os
import re
import subprocess
import sys
import tempfile
from concurrent.futures import ThreadPoolExecutor

from . import build as B

TRANS_PREFIXES = ("v_exp_", "v_log_", "v_rcp_", "v_rsq_", "v_sqrt_", "v_sin_", "v_cos_")
VMEM_PREFIXES = ("global_", "buffer_", "flat_", "scratch_")
MFMA_WAIT = 19
TRANS_WAIT = 1
SGPR_VMEM_WAIT = 5

# the kernel sources that use inline asm
SOURCES = ("uattn_prefill.hip", "uattn_decode.hip", "uattn_backward.hip", "uattn_lm_head.hip")


def _regs(tok: str) -> set:
    tok = tok.strip()
    m = re.match(r"^([vsa])\[(\d+):(\d+)\]$", tok)
    if m:
        return {f"{m.group(1)}{i}" for i in range(int(m.group(2)), int(m.group(3)) + 1)}
    m = re.match(r"^([vsa])(\d+)$", tok)
    if m:
        return {tok}
    if tok == "vcc":
        return {"vcc"}
    return set()


class _Instr:
    __slots__ = ("op", "dst", "srcs", "asm", "line", "text")

    def __init__(self, op, operands, asm, line, text):
        self.op = op
        self.asm = asm
        self.line = line
        self.text = text
        writes_dst = op.startswith(("v_", "s_")) and not op.startswith(
            ("s_cbranch", "s_branch", "s_nop", "s_wait", "s_barrier", "s_setprio", "s_endpgm", "s_cmp", "s_bitcmp",
             "s_sched", "s_sleep", "s_dcache", "s_icache", "s_set", "s_trap", "v_cmpx"))
        if writes_dst and operands:
            self.dst = _regs(operands[0])
            src_ops = operands[1:]
        else:
            self.dst = set()
            src_ops = operands
        self.srcs = set()
        for o in src_ops:
            self.srcs |= _regs(o.split()[0]) if o.strip() else set()


def _parse(text: str):
    """Per function: list of items, each an _Instr or ('label', name)."""
    funcs = {}
    cur = None
    in_asm = False
    for ln, raw in enumerate(text.splitlines(), 1):
        s = raw.strip()
        m = re.match(r"^([A-Za-z_.$][\w.$]*):", s)
        if m and not raw.startswith((" ", "\t")) and not s.startswith(".L"):
            cur = m.group(1)
            funcs[cur] = []
            continue
        if cur is None:
            continue
        if ";;#ASMSTART" in s:
            in_asm = True
            continue
        if ";;#ASMEND" in s:
            in_asm = False
            continue
        if m and s.startswith(".L"):
            funcs[cur].append(("label", m.group(1)))
            continue
        body = s.split(";")[0].strip()
        if not body or body.startswith("."):
            continue
        parts = body.split(None, 1)
        op = parts[0]
        operands = [o for o in parts[1].split(",")] if len(parts) > 1 else []
        funcs[cur].append(_Instr(op, operands, in_asm, ln, body))
    return funcs


def _wait_states(ins: _Instr) -> int:
    if ins.op == "s_nop":
        parts = ins.text.split()
        try:
            return int(parts[1], 0) + 1 if len(parts) > 1 else 1
        except ValueError:
            return 1
    return 1


def _producers(items, idx, regs, budget, label_sites):
    """The nearest writers of regs before items[idx], along fall-through and
    branch predecessors, within `budget` wait states: yields (instr, distance)."""
    stack = [(idx - 1, 0, frozenset(regs))]
    seen = set()
    while stack:
        i, dist, want = stack.pop()
        while i >= 0 and want:
            it = items[i]
            if isinstance(it, tuple):
                for site in label_sites.get(it[1], ()):
                    # continue before the branch instruction, which counts one wait state
                    key = (site, dist, want)
                    if key not in seen and dist + 1 < budget:
                        seen.add(key)
                        stack.append((site - 1, dist + 1, want))
                i -= 1
                continue
            if it.op in ("s_branch", "s_endpgm") or it.op.startswith("s_setpc"):
                break  # nothing falls through into what follows
            hit = it.dst & want
            if hit:
                yield it, dist
                want = want - hit
            dist += _wait_states(it)
            if dist >= budget:
                break
            i -= 1


def scan(text: str):
    """Findings (strings) for one assembly text."""
    findings = []
    for fname, items in _parse(text).items():
        label_sites = {}
        for i, it in enumerate(items):
            if not isinstance(it, tuple) and (it.op.startswith("s_cbranch") or it.op == "s_branch"):
                target = it.text.split()[-1]
                label_sites.setdefault(target, []).append(i)
        for idx, it in enumerate(items):
            if isinstance(it, tuple) or not it.asm:
                continue
            if it.op.startswith("v_") and not it.op.startswith(TRANS_PREFIXES):
                vsrc = {r for r in it.srcs if r.startswith("v")}
                for p, d in _producers(items, idx, vsrc, MFMA_WAIT, label_sites):
                    if p.op.startswith(TRANS_PREFIXES) and d < TRANS_WAIT:
                        findings.append(f"{fname}: line {it.line}: '{it.text}' reads the result of '{p.text}' "
                                        f"with {d} wait states (needs {TRANS_WAIT})")
                    if p.op.startswith("v_mfma") and d < MFMA_WAIT:
                        findings.append(f"{fname}: line {it.line}: '{it.text}' reads the result of '{p.text}' "
                                        f"with {d} wait states (needs up to {MFMA_WAIT})")
            if it.op.startswith(VMEM_PREFIXES):
                ssrc = {r for r in it.srcs if r.startswith("s") or r == "vcc"}
                for p, d in _producers(items, idx, ssrc, SGPR_VMEM_WAIT, label_sites):
                    if p.op.startswith("v_") and d < SGPR_VMEM_WAIT:
                        findings.append(f"{fname}: line {it.line}: '{it.text}' reads an SGPR written by "
                                        f"'{p.text}' with {d} wait states (needs {SGPR_VMEM_WAIT})")
    return findings


def assembly(src: str) -> str:
    """gfx950 device assembly of one kernel source, built with the library's flags."""
    with tempfile.TemporaryDirectory() as tmp:
        out = os.path.join(tmp, os.path.basename(src)[:-4] + ".s")
        cmd = [B.hipcc(), *B.COMMON_FLAGS, *B.PER_FILE_FLAGS.get(os.path.basename(src), []), f"-I{B.INCLUDE}",
               f"-I{B.CSRC}", "--cuda-device-only", "-S", src, "-o", out]
        res = subprocess.run(cmd, capture_output=True, text=True)
        if res.returncode:
            raise RuntimeError(f"assembly of {src} failed:\n{res.stderr[-4000:]}")
        with open(out) as fh:
            return fh.read()


def check(sources=SOURCES):
    """{source: findings} for the kernel sources."""
    paths = [os.path.join(B.CSRC, s) for s in sources]
    with ThreadPoolExecutor(max(1, min(len(paths), os.cpu_count() or 1))) as ex:
        texts = list(ex.map(assembly, paths))
    return {s: scan(t) for s, t in zip(sources, texts)}


def main() -> int:
    bad = 0
    for src, found in check().items():
        print(f"{src}: {len(found)} finding(s)")
        for f in found:
            print("  " + f)
        bad += len(found)
    return 1 if bad else 0


if __name__ == "__main__":
    sys.exit(main())
