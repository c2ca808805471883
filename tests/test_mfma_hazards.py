"""Wait states between MFMA results and the vector instructions that read them
(CPU, needs hipcc).

gfx950 does not interlock a VALU read of a VGPR that an MFMA is still
writing: the code must leave enough independent instructions or s_nop wait
states between the two.  The compiler inserts them, but once missed them on
the path that branches around the attention's key mask: the rescale vote
read the score registers two instructions after the last score MFMA, and
results changed from run to run.  This test compiles the kernel sources to
gfx950 assembly and follows every path (fall-through and branch targets) from
each MFMA; a VALU instruction reading the MFMA's destination within fewer
than 8 wait states (s_nop N counts N + 1) fails it.  Every MFMA in these
kernels needs more than that, so the check catches reads that are far too
early without modelling each instruction's exact requirement.
"""
import os
import re
import shutil
import subprocess

import pytest

from paper_2607_12422_amd import build as b

MIN_WAIT = 8


def _regs(tok):
    m = re.fullmatch(r"([va])\[(\d+):(\d+)\]", tok)
    if m:
        return {f"{m.group(1)}{k}" for k in range(int(m.group(2)), int(m.group(3)) + 1)}
    if re.fullmatch(r"[va]\d+", tok):
        return {tok}
    return set()


def early_reads(asm, limit=MIN_WAIT):
    """(function, mfma line, reader line, wait states) for every VALU read of
    an MFMA destination reached within `limit` wait states on some path."""
    ins, labels, func = [], {}, None
    for i, line in enumerate(asm.splitlines()):
        t = line.split(";")[0].strip()
        if not t:
            continue
        m = re.match(r"^([\w.$]+):$", t)
        if m:
            labels[m.group(1)] = len(ins)
            if not m.group(1).startswith("."):
                func = m.group(1)
            continue
        if t.startswith("."):
            continue
        parts = t.split(None, 1)
        ops = [o.strip() for o in re.split(r",(?![^\[]*\])", parts[1])] if len(parts) > 1 else []
        ins.append((i + 1, parts[0], ops, func))
    found = []
    for k, (ln, op, ops, fn) in enumerate(ins):
        if not op.startswith("v_mfma"):
            continue
        dst = _regs(ops[0])
        stack, seen = [(k + 1, 0)], set()
        while stack:
            j, w = stack.pop()
            if j >= len(ins) or w >= limit or (j, w) in seen:
                continue
            seen.add((j, w))
            ln2, op2, ops2, fn2 = ins[j]
            if fn2 != fn or op2 == "s_endpgm":
                continue
            if op2.startswith("v_") and not op2.startswith("v_mfma") and len(ops2) > 1:
                if set().union(*[_regs(o) for o in ops2[1:]]) & dst:
                    found.append((fn, ln, ln2, w))
            nw = w + (int(ops2[0], 0) + 1 if op2 == "s_nop" else 1)
            if op2.startswith("s_cbranch") or op2 == "s_branch":
                if ops2 and ops2[0] in labels:
                    stack.append((labels[ops2[0]], nw))
                if op2 == "s_branch":
                    continue
            stack.append((j + 1, nw))
    return found


def test_scanner_flags_an_early_read():
    """The scanner itself: a read one wait state after the MFMA on the
    branch-taken path and three on the fall-through path is flagged on both;
    the same read after an s_nop 7 (8 wait states) is not."""
    asm = "\n".join([
        "k:",
        "\tv_mfma_f32_16x16x32_bf16 v[4:7], v[0:3], v[8:11], 0",
        "\ts_cbranch_scc1 .LBB0_2",
        "\tv_add_f32_e32 v20, v21, v22",
        "\tv_add_f32_e32 v20, v21, v22",
        ".LBB0_2:",
        "\tv_max3_f32 v30, v4, v5, v6",
        "\ts_endpgm",
        "k2:",
        "\tv_mfma_f32_16x16x32_bf16 v[4:7], v[0:3], v[8:11], 0",
        "\ts_nop 7",
        "\tv_max3_f32 v30, v4, v5, v6",
        "\ts_endpgm",
    ])
    hits = early_reads(asm)
    assert sorted((h[0], h[3]) for h in hits) == [("k", 1), ("k", 3)]


@pytest.mark.slow
def test_no_valu_reads_an_mfma_result_too_early(tmp_path):
    cc = b.hipcc()
    if not shutil.which(cc) and not os.path.exists(cc):
        pytest.skip("hipcc not available")
    bad = []
    for src in ("pbd_kernels.hip", "pbd_fused.hip"):
        out = tmp_path / (src + ".s")
        cmd = [cc, *b.FLAGS, "--cuda-device-only", "-S", os.path.join(b.CSRC, src), "-o", str(out)]
        r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
        assert r.returncode == 0, r.stdout[-2000:]
        asm = out.read_text()
        assert asm.count("v_mfma") > 100, src
        bad += [(src,) + h for h in early_reads(asm)]
    assert not bad, bad[:10]
