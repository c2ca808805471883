"""GPU parity of the chunked prefill (cfg.prefill_chunk rows per sequence per
pass: the chunk's K/V appended first, chunk-mode attention over the cache,
projections as one GEMM over batch * chunk rows) against the oracle.

The prefill's outputs are the first token (anchor), the lengths and the K/V
cache; the cache is checked through the draft and verify passes that follow.
Tolerances as in the other parity tests: 1e-4 (tiny fp32), 2e-2 (bf16).
"""
import numpy as np
import pytest

import synth
from oracle import model as om

from gpu_harness import GpuRun, decisive

pytestmark = pytest.mark.gpu

TOL32 = 1e-4


def _tiny(D=16):
    cfg = synth.TINY.with_(block=D)
    return cfg, synth.make_weights(cfg, synth.WORKLOADS[0].seed(0))


def _check_after_prefill(g, m, prompts, anchors, tol):
    cfg = m.cfg
    d, dlg = g.draft()
    v, vlg = g.verify(d)
    for b, p in enumerate(prompts):
        empty = [np.zeros((0, cfg.n_kv_heads, cfg.head_dim)) for _ in range(cfg.n_layers)]
        lg, k, vv = m.forward_block(p, 0, empty, empty, causal=True, adapter_on=False, logit_rows=[len(p) - 1])
        if decisive(lg, tol)[0]:
            assert int(np.argmax(lg[0])) == int(anchors[b]), b
        st = om.SeqState(k, vv, int(anchors[b]), tokens=list(p) + [int(anchors[b])])
        _, dl_ref = om.draft(m, st)
        e = float(np.abs(dlg.cpu().numpy()[b] - dl_ref).max())
        assert e <= tol, ("draft", b, e)
        _, vl_ref, _, _ = om.verify(m, st, d.cpu().numpy()[b])
        e = float(np.abs(vlg.cpu().numpy()[b] - vl_ref).max())
        assert e <= tol, ("verify", b, e)


@pytest.mark.parametrize("chunk", [1, 32, 48, 100, 160])
def test_tiny_chunked_prefill_matches_oracle(chunk):
    """Ragged batch (5, 40, 129 tokens): chunk boundaries inside and past the
    prompts, a chunk larger than every prompt, and one row per pass."""
    cfg, w = _tiny()
    lens = [5, 40, 129]
    prompts = synth.make_prompts(cfg, lens, 7)
    g = GpuRun(cfg, w, max_batch=4, max_seq=192, prefill_chunk=chunk)
    anchors = g.prefill(prompts)
    assert list(g.seq_len.cpu().numpy()) == lens
    m = om.OracleModel(w)
    _check_after_prefill(g, m, prompts, anchors, TOL32)
    assert g.status() == 0
    g.close()


def test_chunked_prefill_equals_block_width_prefill():
    """Chunks of 64 rows and the D + 1 row passes give the same first tokens
    and, through the next passes, the same cache (to fp32 rounding)."""
    cfg, w = _tiny()
    prompts = synth.make_prompts(cfg, [150, 77], 21)
    outs = []
    for chunk in (0, 64):
        g = GpuRun(cfg, w, max_batch=2, max_seq=256, prefill_chunk=chunk)
        a = g.prefill(prompts)
        d, dlg = g.draft()
        outs.append((a, dlg.cpu().numpy()))
        g.close()
    assert np.array_equal(outs[0][0], outs[1][0])
    assert np.abs(outs[0][1] - outs[1][1]).max() <= 1e-5


def test_qwen_shape_chunked_prefill_matches_oracle():
    """Qwen3-0.6B shape, bf16, prefix 512 in two 256-row chunks."""
    w_ = synth.WORKLOADS[1]
    cfg = w_.cfg
    w = synth.make_weights(cfg, w_.seed(0))
    lengths, prompts = synth.workload_inputs(w_)
    g = GpuRun(cfg, w, max_batch=1, max_seq=1024, prefill_chunk=256)
    anchors = g.prefill(prompts)
    m = om.OracleModel(w)
    _check_after_prefill(g, m, prompts, anchors, 2e-2)
    assert g.status() == 0
    g.close()
