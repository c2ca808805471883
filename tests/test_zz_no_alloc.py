"""pbd_verify_block_noalloc against pbd_verify_block through the C ABI.

The no-allocation verify runs the same pass with its workspace regions in the
library's static device scratch.  On a model of the Qwen3-0.6B layer shape
(two layers, 4096-token vocabulary) with two sequences of different prefix
lengths, two calls in a row -- batch 2, then batch 1 (a smaller input, so the
second call runs on what the first left in the scratch) -- must give the
verify tokens of pbd_verify_block exactly at decisive rows and its logits
within 2e-2, leave the same cache rows, and raise no status bit.  Both entry
points run in each pass mode of the context (the no-allocation call always
runs one kernel per operator).
"""
import numpy as np
import pytest

import synth

from gpu_harness import GpuRun, decisive

pytestmark = pytest.mark.gpu

TOL = 2e-2


def _cfg():
    return synth.QWEN3_0_6B.with_(n_layers=2, vocab=4096, block=16)


def _verify(g, fn, batch):
    W, V = g.cfg.width, g.cfg.vocab
    v = g.zeros(batch, W)
    lg = g.zeros(batch, W, V, dtype=g.torch.float32)
    fn(g.seq_len[:batch], g.anchor[:batch], g.d[:batch].contiguous(), v, lg)
    g.torch.cuda.synchronize()
    return v.cpu().numpy(), lg.cpu().numpy()


def _compare(ref, got, what):
    (v0, l0), (v1, l1) = ref, got
    err = float(np.abs(l0 - l1).max())
    print(f"{what}: logits max-abs {err:.2e}")
    assert err <= TOL, (what, err)
    for b in range(v0.shape[0]):
        dec = decisive(l0[b], TOL)
        assert np.array_equal(v0[b][dec], v1[b][dec]), (what, b, v0[b], v1[b])


@pytest.mark.parametrize("mode", [1, 0])
def test_noalloc_verify_matches_verify_twice(mode):
    cfg = _cfg()
    w = synth.make_weights(cfg, 7100)
    prompts = synth.make_prompts(cfg, [144, 64], 7101)     # block rows start a 16-position cache block
    g = GpuRun(cfg, w, max_batch=2, max_seq=400)
    g.eng.pbd_set_pass_mode(mode)
    g.prefill(prompts)
    g.d, _ = g.draft()
    # cache as [K/V][layer][sequence][KV head][16-position block][16 * head_dim]
    # (bf16; the element order inside a block is the kernels' own)
    nblk = (400 + 15) // 16
    kv = g.eng.kv.view(g.torch.bfloat16).view(2, cfg.n_layers, 2, cfg.n_kv_heads, nblk, 16 * cfg.head_dim)
    t = g.seq_len.cpu().numpy()
    assert np.all(t % 16 == 0)
    for batch in (2, 1):
        ref = _verify(g, g.eng.pbd_verify_block, batch)
        kv_ref = kv.clone()
        for b in range(batch):                  # the no-allocation call must write the block rows again
            kv[:, :, b, :, t[b] // 16:(t[b] + cfg.width + 15) // 16] = 0
        got = _verify(g, g.eng.pbd_verify_block_noalloc, batch)
        _compare(ref, got, f"mode {mode} batch {batch}")
        kd = float((kv.float() - kv_ref.float()).abs().max())
        print(f"mode {mode} batch {batch}: cache max-abs {kd:.2e}")
        assert kd <= TOL
    assert g.status() == 0
    g.close()


def test_noalloc_verify_rejects_a_context_beyond_the_scratch():
    from paper_2607_12422_amd import binding as bd
    cfg = _cfg()
    w = synth.make_weights(cfg, 7200)
    g = GpuRun(cfg, w, max_batch=4, max_seq=1100)   # about 39 MiB of pass workspace
    s, d, v = g.zeros(4), g.zeros(4, cfg.block), g.zeros(4, cfg.width)
    with pytest.raises(bd.PbdError) as ei:
        g.eng.pbd_verify_block_noalloc(s, s, d, v)
    assert ei.value.code == bd.PBD_ERR_CAPACITY
    g.close()
