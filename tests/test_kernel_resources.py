"""Compile-time resource check of the hot-path kernels (CPU, needs hipcc).

A register array indexed with a run-time value, or a register budget that
overflows, puts per-lane data in scratch memory, which turns every access into
a global memory round trip.  The kernels of the Qwen3-shape passes (the persistent
layer stack; bf16 with split operands; projection GEMMs at every LoRA rank up to 64; attention with
head_dim 128 and up to three 16-row query tiles, and the prefix splits of
four or five) and every projection GEMM of
the fp32 model must use no scratch at all.
"""
import os
import re
import shutil
import subprocess

import pytest

from paper_2607_12422_amd import build as b

HOT = [
    # projection GEMMs (bf16 value + residual operands; fp32), LoRA rank <= 64
    r"_ZN3pbd7k_fgemmIDF16bLi\d+ELi\d+ELb1ELi[0-4]EEEvNS_9FGemmArgsE",
    r"_ZN3pbd7k_fgemmIfLi\d+ELi\d+ELb0ELi[0-4]EEEvNS_9FGemmArgsE",
    r"_ZN3pbd6k_attnIDF16bLi128ELi[123]EEEvNS_8AttnArgsE",            # attention, G*W <= 48 query rows
    r"_ZN3pbd11k_attn_rowsILi[45]EEEvNS_8AttnArgsE",                  # prefix splits, 49..80 query rows
    r"_ZN3pbd8k_lmheadIDF16bLb1ELb[01]EEEvNS_9FGemmArgsE",            # LM head (with / without confidence)
    r"_ZN3pbd9k_combineIDF16bLi\d+EEEvNS_11CombineArgsE",
    r"_ZN3pbd10k_assembleIDF16bEEvNS_12AssembleArgsE",
    r"_ZN3pbd8k_argmaxILi(1|8)EEEvNS_10ArgmaxArgsE",
    r"_ZN3pbd8k_acceptENS_10AcceptArgsE",
    r"_ZN3pbd8k_remaskENS_10RemaskArgsE",
    # prefill chunks
    r"_ZN3pbd10k_gemm_bigIDF16bLb[01]ELi[24]ELb[01]EEEvNS_11BigGemmArgsE",
    r"_ZN3pbd9k_kvwriteIDF16bLi128EEEvNS_11KVWriteArgsE",
    r"_ZN3pbd13k_gather_lastIDF16bEEvNS_10GatherArgsE",
    # the persistent batch-1 layer stack (adapter on / off)
    r"_ZN3pbd2fz7k_fusedILb[01]EEEvNS_9FusedArgsE",
]


@pytest.mark.slow
def test_hot_kernels_use_no_scratch(tmp_path):
    cc = b.hipcc()
    if not shutil.which(cc) and not os.path.exists(cc):
        pytest.skip("hipcc not available")
    out = ""
    for src in ("pbd_kernels.hip", "pbd_fused.hip"):
        cmd = [cc, *b.FLAGS, "-c", os.path.join(b.CSRC, src), "-o", str(tmp_path / (src + ".o")),
               "-Rpass-analysis=kernel-resource-usage"]
        out += subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True).stdout
    usage = {}
    name = None
    for line in out.splitlines():
        m = re.search(r"Function Name: (\S+)", line)
        if m:
            name = m.group(1)
        m = re.search(r"ScratchSize \[bytes/lane\]: (\d+)", line)
        if m and name:
            usage[name] = int(m.group(1))
    assert usage, out[-2000:]
    seen = 0
    for pat in HOT:
        names = [n for n in usage if re.fullmatch(pat, n)]
        assert names, f"no kernel matches {pat}"
        for n in names:
            seen += 1
            assert usage[n] == 0, f"{n} uses {usage[n]} bytes of scratch per lane"
    assert seen >= 15
