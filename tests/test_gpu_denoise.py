"""GPU parity of multi-step drafting (pbd_draft_block_denoise) against the oracle.

The oracle follows the GPU pass by pass (gpu_harness.check_denoise): at each
pass it runs on the block the GPU had, checks the confidences of the positions
the GPU fixed, their tokens at decisive rows, and the choice of positions
(exact where the oracle's confidence gap at the cut is decisive, else valid
within the tolerance).  Tolerances: 1e-4 on logits for the fp32 tiny model,
2e-2 for the bf16 Qwen3-0.6B shape.
"""
import numpy as np
import pytest

import synth
from oracle import model as om

from gpu_harness import GpuRun, check_denoise

pytestmark = pytest.mark.gpu

TOL32 = 1e-4


def _tiny(D=16):
    cfg = synth.TINY.with_(block=D)
    return cfg, synth.make_weights(cfg, synth.WORKLOADS[0].seed(0))


@pytest.mark.parametrize("k", [2, 3, 16])
def test_tiny_denoise_matches_oracle(k):
    cfg, w = _tiny()
    lengths, prompts = synth.workload_inputs(synth.WORKLOADS[0])
    g = GpuRun(cfg, w, max_batch=1, max_seq=256)
    g.prefill(prompts)
    m = om.OracleModel(w)
    st = om.prefill(m, prompts[0])
    d, conf, fixed, lg = g.denoise(k)
    worst = check_denoise(m, st, d.cpu().numpy()[0], conf.cpu().numpy()[0], fixed.cpu().numpy()[0],
                          lg.cpu().numpy()[0], k, TOL32, what=f"k={k}")
    print(f"tiny k={k}: worst confidence error {worst:.2e}")
    # the k passes leave the KV cache alone: the one-step draft and the verify
    # that follow still match the oracle's untouched state
    d1, dlg = g.draft()
    _, dl_ref = om.draft(m, st)
    assert np.abs(dlg.cpu().numpy()[0] - dl_ref).max() <= TOL32
    v, vlg = g.verify(d1)
    _, vl_ref, _, _ = om.verify(m, st, d1.cpu().numpy()[0])
    assert np.abs(vlg.cpu().numpy()[0] - vl_ref).max() <= TOL32
    assert g.status() == 0
    g.close()


def test_one_pass_is_the_one_step_draft():
    """n_steps = 1 gives pbd_draft_block's tokens and logits, bit for bit."""
    cfg, w = _tiny()
    lengths, prompts = synth.workload_inputs(synth.WORKLOADS[0])
    g = GpuRun(cfg, w, max_batch=1, max_seq=256)
    g.prefill(prompts)
    d0, lg0 = g.draft()
    d1, conf, fixed, lg1 = g.denoise(1)
    assert g.torch.equal(d0, d1) and g.torch.equal(lg0, lg1)
    assert bool((fixed == 1).all())
    m = om.OracleModel(w)
    st = om.prefill(m, prompts[0])
    check_denoise(m, st, d1.cpu().numpy()[0], conf.cpu().numpy()[0], fixed.cpu().numpy()[0],
                  lg1.cpu().numpy()[0], 1, TOL32, what="k=1")
    g.close()


@pytest.mark.parametrize("k", [2, 5])
def test_tiny_ragged_batch_denoise(k):
    """Three sequences of different lengths (51 block rows: the LM head runs
    as the tiled GEMM with the argmax epilogue)."""
    cfg, w = _tiny()
    lens = [5, 40, 129]
    prompts = synth.make_prompts(cfg, lens, 7)
    g = GpuRun(cfg, w, max_batch=4, max_seq=192)
    g.prefill(prompts)
    d, conf, fixed, lg = g.denoise(k)
    m = om.OracleModel(w)
    d, conf, fixed, lg = (x.cpu().numpy() for x in (d, conf, fixed, lg))
    for b, p in enumerate(prompts):
        st = om.prefill(m, p)
        check_denoise(m, st, d[b], conf[b], fixed[b], lg[b], k, TOL32, what=f"seq {b} k={k}")
    g.close()


def test_tiny_batch16_denoise():
    """Sixteen sequences (272 block rows): the final argmax takes eight rows
    per work-group, merging each row's confidence partials in another order
    than at fewer rows; tokens, confidences and fixing order against the
    oracle."""
    cfg, w = _tiny()
    lens = [5 + 9 * i for i in range(16)]
    prompts = synth.make_prompts(cfg, lens, 17)
    g = GpuRun(cfg, w, max_batch=16, max_seq=192)
    g.prefill(prompts)
    d, conf, fixed, lg = g.denoise(3)
    m = om.OracleModel(w)
    d, conf, fixed, lg = (x.cpu().numpy() for x in (d, conf, fixed, lg))
    for b, p in enumerate(prompts):
        st = om.prefill(m, p)
        check_denoise(m, st, d[b], conf[b], fixed[b], lg[b], 3, TOL32, what=f"seq {b} of 16")
    g.close()


def test_denoise_rejects_bad_step_counts():
    from paper_2607_12422_amd.binding import PbdError
    cfg, w = _tiny(4)
    lengths, prompts = synth.workload_inputs(synth.WORKLOADS[0])
    g = GpuRun(cfg, w, max_batch=1, max_seq=256)
    g.prefill(prompts)
    for bad in (0, 5):
        with pytest.raises(PbdError):
            g.denoise(bad)
    d, conf, fixed, lg = g.denoise(4)          # one position per pass
    assert sorted(fixed.cpu().numpy()[0].tolist()) == [1, 2, 3, 4]
    g.close()


def test_qwen_shape_two_step_denoise_matches_oracle():
    """Qwen3-0.6B shape, bf16, prefix 512: the two-step draft of the ablation."""
    w_ = synth.WORKLOADS[1]
    cfg = w_.cfg
    w = synth.make_weights(cfg, w_.seed(0))
    lengths, prompts = synth.workload_inputs(w_)
    g = GpuRun(cfg, w, max_batch=1, max_seq=1024)
    g.prefill(prompts)
    d, conf, fixed, lg = g.denoise(2)
    m = om.OracleModel(w)
    st = om.prefill(m, prompts[0])
    worst = check_denoise(m, st, d.cpu().numpy()[0], conf.cpu().numpy()[0], fixed.cpu().numpy()[0],
                          lg.cpu().numpy()[0], 2, 2e-2, what="qwen k=2")
    print(f"qwen k=2: worst confidence error {worst:.4f}")
    assert g.status() == 0
    g.close()
