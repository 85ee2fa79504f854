"""Audit of the block-scaled GEMM's hand-placed MFMA wait states, on the code the
compiler emits (CPU only: hipcc compiles every GEMM source to gfx950 assembly).

The GEMM issues v_mfma_scale_f32_16x16x128_f8f6f4 as inline assembly with the
accumulator tied (gemm_mx.h, mma / mma_drain), so the compiler's hazard
recognizer does not see these instructions.  The wait states they need are
written by hand: two before each MFMA (a VALU write of an operand just before
it) and a 24-state drain before any other instruction touches the
accumulators.  This test walks the control-flow graph of every kernel that
contains the instruction and checks, for every path:

* every VGPR an MFMA reads (operands and scale bytes) was last written by a
  VALU instruction at least 2 wait states earlier;
* no instruction other than an MFMA reads or writes an accumulator register
  within MIN_ACC wait states of an MFMA that read or wrote it;
* MFMAs that accumulate into the same registers back to back use the same
  operand formats (cbsz / blgp), the case whose forwarding needs no wait
  states; a change of formats needs MIN_ACC states in between.

Wait states are counted as the hazard rules count them: s_nop N is N + 1 and
any other instruction in between is 1 (a lower bound on its issue time).
MIN_ACC = 19 is the bound the kernel is written to (a 16x16x128 block-scaled
MFMA needs at most 19 before another instruction uses its result); the drain
provides 24.  In the current code the epilogue reads the accumulators in the
order they were last written, so the nearest read comes well after the drain.
"""
import os
import re
import shutil
import subprocess
import tempfile
from concurrent.futures import ProcessPoolExecutor

import pytest

from paper_2110_15456_amd import build as B

MFMA = "v_mfma_scale_f32_16x16x128_f8f6f4"
MIN_VALU = 2
MIN_ACC = 19
CAP = 64  # distances beyond this are "far"

_REG = re.compile(r"\b([av])(?:\[(\d+):(\d+)\]|(\d+)(?!\w))")
_BRANCH = re.compile(r"^s_(c?branch)\w*\s+(\.L\w+)")


def _regs(text):
    """(kind, index) of every register named in an operand string."""
    out = []
    for m in _REG.finditer(text):
        kind = m.group(1)
        if m.group(4) is not None:
            out.append((kind, int(m.group(4))))
        else:
            out.extend((kind, i) for i in range(int(m.group(2)), int(m.group(3)) + 1))
    return out


def _operands(line):
    parts = line.split(None, 1)
    return parts[0], (parts[1] if len(parts) > 1 else "")


def _kernels(asm):
    """{name: [instruction lines and labels]} of the kernels that issue MFMA."""
    kernels, cur, name = {}, None, None
    for raw in asm.splitlines():
        m = re.match(r"^(_Z\w+):", raw)
        if m:
            name, cur = m.group(1), []
            continue
        if cur is None:
            continue
        s = raw.strip()
        if not s or s.startswith(";") or (s.startswith(".") and not re.match(r"^\.L\w+:", s)):
            continue
        cur.append(s.split(";")[0].strip())
        if s.startswith("s_endpgm"):
            if any(MFMA in x for x in cur):
                kernels[name] = cur
            cur, name = None, None
    return kernels


def _blocks(lines):
    """Basic blocks: (label or None, instructions, successor labels, falls through)."""
    blocks, cur_label, cur = [], None, []

    def close(fall):
        blocks.append([cur_label, list(cur), [], fall])

    for s in lines:
        m = re.match(r"^(\.L\w+):", s)
        if m:
            if cur or cur_label is not None:
                close(True)
            cur_label, cur = m.group(1), []
            continue
        cur.append(s)
        b = _BRANCH.match(s)
        if b or s.startswith("s_endpgm") or s.startswith("s_setpc"):
            close(bool(b) and b.group(1) == "cbranch")
            if b:
                blocks[-1][2].append(b.group(2))
            cur_label, cur = None, []
    if cur or cur_label is not None:
        close(False)
    return blocks


def _cost(ins):
    op = ins.split(None, 1)[0]
    if op == "s_nop":
        return int(ins.split()[1], 0) + 1
    return 1


def _decode(ins):
    """(is_mfma, cost, mnemonic, registers, MFMA destination or VOP destination VGPRs, MFMA formats)."""
    op, rest = _operands(ins)
    if op == MFMA:
        regs = _regs(rest.split(" op_sel")[0].split(" cbsz")[0])
        fmt = " ".join(re.findall(r"(?:cbsz|blgp):\d", rest)) or "cbsz:0 blgp:0"
        return True, 1, op, regs, _regs(rest.split(",")[0]), fmt
    regs = _regs(rest)
    dst = ()
    if op.startswith("v_") and regs and regs[0][0] == "v":
        dst = tuple(r for r in _regs(rest.split(",")[0]) if r[0] == "v")  # VOP destination
    return False, _cost(ins), op, regs, dst, None


def _audit_kernel(lines):
    """Violations found in one kernel: list of strings."""
    blocks = _blocks(lines)
    code = [[_decode(x) for x in b[1]] for b in blocks]
    index = {b[0]: i for i, b in enumerate(blocks) if b[0] is not None}
    preds = [[] for _ in blocks]
    for i, (label, ins, succ, fall) in enumerate(blocks):
        for t in succ:
            if t in index:
                preds[index[t]].append(i)
        if fall and i + 1 < len(blocks):
            preds[i + 1].append(i)
    # exit states: {reg: distance} for VALU-written VGPRs and MFMA-touched
    # AGPRs (with the formats of that MFMA)
    exit_v = [dict() for _ in blocks]
    exit_a = [dict() for _ in blocks]
    violations = set()

    def walk(i, record):
        ent_v, ent_a = {}, {}
        for p in preds[i]:
            for r, d in exit_v[p].items():
                ent_v[r] = min(ent_v.get(r, CAP), d)
            for r, (d, fmt) in exit_a[p].items():
                if r not in ent_a or d < ent_a[r][0]:
                    ent_a[r] = (d, fmt)
        now = 0
        tv = {r: -d for r, d in ent_v.items()}
        ta = {r: (-d, fmt) for r, (d, fmt) in ent_a.items()}
        for is_mfma, cost, op, regs, dst, fmt in code[i]:
            if is_mfma:
                if record:
                    for r in regs:
                        if r[0] == "v" and r in tv and now - tv[r] < MIN_VALU:
                            violations.add("VALU write of %s%d %d states before an MFMA read" % (r[0], r[1], now - tv[r]))
                    for r in dst:
                        if r in ta and ta[r][1] != fmt and now - ta[r][0] < MIN_ACC:
                            violations.add("accumulator %s%d chained across formats %s -> %s after %d states" %
                                           (r[0], r[1], ta[r][1], fmt, now - ta[r][0]))
                now += cost
                for r in regs:
                    if r[0] == "a":
                        ta[r] = (now, fmt)
                continue
            if record:
                for r in regs:
                    if r[0] == "a" and r in ta and now - ta[r][0] < MIN_ACC:
                        violations.add("%s touches %s%d %d states after an MFMA" % (op, r[0], r[1], now - ta[r][0]))
            now += cost
            for r in dst:
                tv[r] = now
        new_v = {r: now - t for r, t in tv.items() if now - t < CAP}
        new_a = {r: (now - t, f) for r, (t, f) in ta.items() if now - t < CAP}
        changed = new_v != exit_v[i] or new_a != exit_a[i]
        exit_v[i], exit_a[i] = new_v, new_a
        return changed

    for _ in range(len(blocks) + 2):  # distances only shrink: a fixed point
        if not any([walk(i, False) for i in range(len(blocks))]):
            break
    for i in range(len(blocks)):
        walk(i, True)
    return sorted(violations)


def _audit_source(src):
    """Compile one GEMM source to gfx950 assembly (the library's flags) and
    audit its kernels: (kernels, MFMA instructions, {kernel: violations})."""
    flags = [f for f in B.HIPFLAGS if f not in ("-fPIC",)]
    with tempfile.TemporaryDirectory() as d:
        out = os.path.join(d, "k.s")
        cmd = [os.path.join(B.ROCM, "bin", "hipcc"), *flags, *B.SOURCE_FLAGS.get(os.path.basename(src), []),
               "--cuda-device-only", "-S", "-o", out, src]
        res = subprocess.run(cmd, capture_output=True, text=True)
        if res.returncode != 0:
            raise RuntimeError(res.stderr[-2000:])
        with open(out) as f:
            kernels = _kernels(f.read())
    bad = {}
    nmfma = 0
    for name, lines in kernels.items():
        nmfma += sum(1 for x in lines if x.startswith(MFMA))
        v = _audit_kernel(lines)
        if v:
            bad[name] = v[:5]
    return len(kernels), nmfma, bad


def test_audit_finds_planted_hazards():
    """The checker itself: a VALU write right before an MFMA, an accumulator
    read right after one, and a format change on a chained accumulator are
    each reported; the same code with the wait states is clean."""
    ok = ["v_mov_b32_e32 v2, v9", "s_nop 1",
          MFMA + " a[0:3], v[2:7], v[8:13], a[0:3], v20, v21 op_sel_hi:[0,0,0] cbsz:2 blgp:2",
          "s_nop 7", "s_nop 7", "s_nop 7", "v_accvgpr_read_b32 v30, a1", "s_endpgm"]
    assert _audit_kernel(ok) == []
    no_nop = [x for x in ok if x != "s_nop 1"]
    assert any("VALU write of v2" in v for v in _audit_kernel(no_nop))
    short_drain = ok[:3] + ["s_nop 7"] + ok[6:]
    assert any("touches a1" in v for v in _audit_kernel(short_drain))
    mixed = ok[:3] + ["s_nop 1", MFMA + " a[0:3], v[2:5], v[8:13], a[0:3], v20, v21 op_sel_hi:[0,0,0] cbsz:4 blgp:2"] + ok[3:]
    assert any("chained across formats" in v for v in _audit_kernel(mixed))
    # across a loop back edge: the read at the top of the loop follows the
    # MFMA at its bottom
    loop = [".LBB0_1:", "v_accvgpr_read_b32 v30, a1", "s_nop 1",
            MFMA + " a[0:3], v[2:7], v[8:13], a[0:3], v20, v21 op_sel_hi:[0,0,0] cbsz:2 blgp:2",
            "s_cbranch_scc1 .LBB0_1", "s_endpgm"]
    assert any("touches a1" in v for v in _audit_kernel(loop))


@pytest.mark.skipif(shutil.which(os.path.join(B.ROCM, "bin", "hipcc")) is None, reason="hipcc not available")
def test_gemm_kernels_respect_mfma_wait_states():
    srcs = sorted(os.path.join(B.CSRC, f) for f in os.listdir(B.CSRC) if f.startswith("gemm_mx") and f.endswith(".hip"))
    assert srcs
    with ProcessPoolExecutor(max_workers=max(1, min(8, os.cpu_count() or 1))) as ex:
        results = list(ex.map(_audit_source, srcs))
    nkernels = sum(r[0] for r in results)
    nmfma = sum(r[1] for r in results)
    bad = {k: v for r in results for k, v in r[2].items()}
    print("audited %d kernels, %d MFMA instructions" % (nkernels, nmfma))
    assert nkernels >= 100 and nmfma > 10000
    assert not bad, bad
