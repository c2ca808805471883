"""Run-to-run determinism of the passes (GPU, through the C ABI).

Every cross-work-group reduction of the HIP path sums in a fixed order: the
split-K residual GEMMs add their K slices in slice order, the attention merge
takes the split-KV partials in split order, the persistent pass adds waves,
groups and splits in index order, the argmax breaks ties by the lowest token
id.  Running the same draft and verify twice on the same state
must therefore give bit-identical logits, tokens and cache rows.  Checked at
batch 1 in both pass modes (the persistent pass; the weight-streaming GEMMs
with their split-K handoff) and at batch 8 (128+ rows: the large-M path), on
the Qwen3-0.6B layer shape with two layers, and on the full Qwen3-0.6B shape
at batch 1.
"""
import numpy as np
import pytest

import synth

from gpu_harness import GpuRun

pytestmark = pytest.mark.gpu


def _twice(g, reps=3):
    outs = []
    for _ in range(reps):
        d, dlg = g.draft()
        v, vlg = g.verify(d)
        outs.append((d.clone(), dlg.clone(), v.clone(), vlg.clone(), g.eng.kv.clone()))
    g.torch.cuda.synchronize()
    return outs


def _check_all_equal(outs, what):
    t = outs[0]
    for r, o in enumerate(outs[1:], 1):
        for i, name in enumerate(("draft", "draft logits", "verify", "verify logits", "kv cache")):
            assert o[i].shape == t[i].shape
            assert bool((o[i] == t[i]).all()), f"{what}: repetition {r} differs in {name}"


@pytest.mark.parametrize("batch,mode", [(1, 0), (1, 1), (8, 0)])
def test_two_layer_qwen_shape_is_deterministic(batch, mode):
    """Batch 1 in pass mode 0 runs the persistent pass, in mode 1 the skinny
    GEMMs with the split-K handoff; batch 8 runs the large-M path."""
    cfg = synth.QWEN3_0_6B.with_(n_layers=2, vocab=4096)
    w = synth.make_weights(cfg, 5100 + batch)
    lengths = [60 + 37 * b for b in range(batch)]
    prompts = synth.make_prompts(cfg, lengths, 5200 + batch)
    g = GpuRun(cfg, w, max_batch=batch, max_seq=max(lengths) + 2 * cfg.width)
    g.eng.pbd_set_pass_mode(mode)
    g.prefill(prompts)
    outs = _twice(g)
    assert g.status() == 0
    _check_all_equal(outs, f"two-layer Qwen shape, batch {batch}, pass mode {mode}")
    g.close()


@pytest.mark.slow
def test_qwen_shape_batch1_is_deterministic():
    w_ = synth.WORKLOADS[1]
    cfg = w_.cfg
    w = synth.make_weights(cfg, w_.seed(0))
    lengths, prompts = synth.workload_inputs(w_)
    g = GpuRun(cfg, w, max_batch=1, max_seq=1024)
    g.prefill(prompts)
    outs = _twice(g)
    assert g.status() == 0
    _check_all_equal(outs, "Qwen3-0.6B shape, batch 1, prefix 512")
    g.close()
