"""GPU parity of the skinny projection GEMM at LoRA ranks 32, 48 and 64.

Batches of one to three sequences keep every pass below the large-M path, so
the adapter runs inside the weight-streaming GEMM with two to four 16-row
shrink tiles per source matrix (App. A.2 fixes r = 16; the larger ranks are
those of the batch-8 and batch-32 workloads).  Each sequence's draft and
verify logits are compared with the oracle: max-abs 1e-4 for the fp32 model,
2e-2 for bf16; token ids equal at decisive rows.  The bf16 model has the
Qwen3-0.6B layer shape with two layers and a 4096-token vocabulary, so that
the float64 oracle finishes in seconds.
"""
import numpy as np
import pytest

import synth
from oracle import model as om

from gpu_harness import GpuRun, decisive

pytestmark = pytest.mark.gpu


def _check(gpu_logits, gpu_tokens, ref_logits, rows, tol, exclude=None, what=""):
    err = float(np.abs(gpu_logits - ref_logits).max())
    print(f"{what}: max-abs {err:.2e}")
    assert err <= tol, (what, err)
    lg = ref_logits[rows].copy()
    dec = decisive(lg, tol, exclude)
    if exclude is not None:
        lg[:, exclude] = -np.inf
    ref = np.argmax(lg, axis=-1)
    assert np.all(gpu_tokens[dec] == ref[dec]), what


def _oracle_prefill(m, prompt, gpu_anchor, tol):
    """Oracle prefill continued with the GPU's first token, which must equal
    the oracle's where the oracle's last-row margin is decisive."""
    cfg = m.cfg
    empty = [np.zeros((0, cfg.n_kv_heads, cfg.head_dim)) for _ in range(cfg.n_layers)]
    lg, k, v = m.forward_block(prompt, 0, empty, empty, causal=True, adapter_on=False,
                               logit_rows=[len(prompt) - 1])
    if decisive(lg, tol)[0]:
        assert int(np.argmax(lg[0])) == int(gpu_anchor)
    return om.SeqState(k, v, int(gpu_anchor), tokens=list(prompt) + [int(gpu_anchor)],
                       generated=[int(gpu_anchor)])


def _run(cfg, tol, batch, seed):
    w = synth.make_weights(cfg, seed)
    lengths = [40 + 23 * b for b in range(batch)]
    prompts = synth.make_prompts(cfg, lengths, seed + 1)
    g = GpuRun(cfg, w, max_batch=batch, max_seq=max(lengths) + 2 * cfg.width)
    anchors = g.prefill(prompts)
    d, dlg = g.draft()
    v, vlg = g.verify(d)
    assert g.status() == 0
    m = om.OracleModel(w)
    d_np, v_np, dlg_np, vlg_np = d.cpu().numpy(), v.cpu().numpy(), dlg.cpu().numpy(), vlg.cpu().numpy()
    for b in range(batch):
        st = _oracle_prefill(m, prompts[b], anchors[b], tol)
        _, dl_ref = om.draft(m, st)
        _check(dlg_np[b], d_np[b], dl_ref, slice(1, None), tol, exclude=cfg.mask_id,
               what=f"r={cfg.lora_rank} B={batch} seq {b} draft")
        _, vl_ref, _, _ = om.verify(m, st, d_np[b])
        _check(vlg_np[b], v_np[b], vl_ref, slice(None), tol, what=f"r={cfg.lora_rank} B={batch} seq {b} verify")
    g.close()


@pytest.mark.parametrize("rank", [32, 64])
@pytest.mark.parametrize("batch", [1, 3])
def test_fp32_high_rank_adapter_matches_oracle(rank, batch):
    cfg = synth.TINY.with_(lora_rank=rank, lora_alpha=2.0 * rank)
    _run(cfg, 1e-4, batch, 4100 + rank + batch)


@pytest.mark.parametrize("rank,batch", [(32, 1), (32, 3), (48, 2), (64, 1), (64, 3)])
def test_bf16_high_rank_adapter_matches_oracle(rank, batch):
    cfg = synth.QWEN3_0_6B.with_(n_layers=2, vocab=4096, lora_rank=rank, lora_alpha=2.0 * rank)
    _run(cfg, 2e-2, batch, 4200 + rank + batch)
