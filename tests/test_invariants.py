"""Method-level invariants of the oracle (tiny model, float64).

* losslessness: whatever the drafts, the committed tokens are exactly the
  verifier's greedy decoding (the exact greedy-output audit of Tab. HF
  diagnostics; App. A.1 exact greedy matching);
* the adapter: with B = 0 the adapter-on pass equals the adapter-off pass;
* the masks: at D = 0 the draft and verify masks coincide; with a causal
  override the draft of [anchor, mask x D] equals the verify of the same block;
* the cache: after any forced acceptance the cached K/V equal a fresh prefill
  of the committed tokens; forcing n = 0 every round is plain greedy decoding.
"""
import numpy as np
import pytest

import synth
from oracle import brute
from oracle import model as om


def _tiny(D=4, seed=0, zero_b=False):
    cfg = synth.TINY.with_(block=D)
    w = synth.make_weights(cfg, seed, zero_lora_b=zero_b)
    return w, om.OracleModel(w)


def test_verify_predictions_are_greedy_next_tokens():
    w, m = _tiny(D=4)
    prompt = synth.make_prompts(m.cfg, [6], 21)[0]
    st = om.prefill(m, prompt)
    drafts = np.array([5, 77, 1023, 9], dtype=np.int32)
    p, _, _, _ = om.verify(m, st, drafts)
    seq = list(prompt) + [st.anchor]
    for j in range(len(drafts) + 1):
        assert p[j] == brute.greedy_decode(w, seq + [int(x) for x in drafts[:j]], 1)[0]


@pytest.mark.parametrize("correct", [4, 2, 0])
def test_scripted_drafts_accept_exactly_the_matching_prefix(correct):
    w, m = _tiny(D=4)
    prompt = synth.make_prompts(m.cfg, [5], 22)[0]
    st = om.prefill(m, prompt)
    greedy = brute.greedy_decode(w, list(prompt) + [st.anchor], 5)
    drafts = np.array(greedy[:4], dtype=np.int32)
    if correct < 4:
        drafts[correct] = (drafts[correct] + 1) % (m.cfg.vocab - 1)
    p, _, k, v = om.verify(m, st, drafts)
    n, out = om.accept(drafts, p)
    assert n == correct
    assert out == greedy[:correct + 1]


def test_loop_output_equals_greedy_decoding_for_any_drafts():
    """The exact greedy audit: a loop fed partly-correct drafts commits exactly
    the greedy continuation."""
    w, m = _tiny(D=4)
    prompt = synth.make_prompts(m.cfg, [5], 23)[0]
    budget = 14
    ref = brute.greedy_decode(w, prompt, budget)
    st = om.prefill(m, prompt)
    rng = np.random.default_rng(0)
    ns = []
    while len(st.generated) < budget:
        # a drafter that knows the reference continuation but corrupts one slot
        pos = len(st.generated)
        cont = ref[pos:pos + 4] + [0] * 4
        drafts = np.array(cont[:4], dtype=np.int32)
        bad = rng.integers(0, 5)
        if bad < 4:
            drafts[bad] = (drafts[bad] + 1) % (m.cfg.vocab - 1)
        p, _, k, v = om.verify(m, st, drafts)
        n, out = om.accept(drafts, p)
        om.commit(st, n, out, k, v)
        ns.append(n)
    assert st.generated[:budget] == ref
    assert max(ns) > 0          # acceptance was exercised


def test_real_drafts_loop_is_lossless():
    w, m = _tiny(D=4)
    prompt = synth.make_prompts(m.cfg, [5], 24)[0]
    gen, rounds, _ = om.generate(m, prompt, 8)
    assert gen == brute.greedy_decode(w, prompt, 8)


def test_forced_zero_acceptance_is_greedy_decoding():
    w, m = _tiny(D=4)
    prompt = synth.make_prompts(m.cfg, [5], 25)[0]
    gen, rounds, _ = om.generate(m, prompt, 6, forced=[0] * 6)
    assert gen == brute.greedy_decode(w, prompt, 6)
    assert rounds == [0] * 5


def test_zero_lora_b_makes_adapter_a_no_op():
    _, m = _tiny(D=4, zero_b=True)
    prompt = synth.make_prompts(m.cfg, [9], 26)[0]
    st = om.prefill(m, prompt)
    d_on, lg_on = om.draft(m, st, adapter_on=True)
    d_off, lg_off = om.draft(m, st, adapter_on=False)
    np.testing.assert_array_equal(lg_on, lg_off)
    np.testing.assert_array_equal(d_on, d_off)


def test_draft_with_causal_override_equals_verify_of_mask_block():
    _, m = _tiny(D=4, zero_b=True)
    prompt = synth.make_prompts(m.cfg, [9], 27)[0]
    st = om.prefill(m, prompt)
    _, lg_d = om.draft(m, st, adapter_on=True, causal=True)
    _, lg_v, _, _ = om.verify(m, st, [m.cfg.mask_id] * 4)
    np.testing.assert_array_equal(lg_d, lg_v)


def test_block_masks_differ_without_override():
    _, m = _tiny(D=4, zero_b=True)
    prompt = synth.make_prompts(m.cfg, [9], 27)[0]
    st = om.prefill(m, prompt)
    _, lg_d = om.draft(m, st)
    _, lg_v, _, _ = om.verify(m, st, [m.cfg.mask_id] * 4)
    assert np.abs(lg_d[:-1] - lg_v[:-1]).max() > 1e-6


def test_width_one_masks_coincide():
    _, m = _tiny(D=0, zero_b=True)
    prompt = synth.make_prompts(m.cfg, [9], 28)[0]
    st = om.prefill(m, prompt)
    _, lg_d = om.draft(m, st)
    p, lg_v, _, _ = om.verify(m, st, [])
    np.testing.assert_array_equal(lg_d, lg_v)
    n, out = om.accept([], p)
    assert n == 0 and out == [int(p[0])]


def test_cache_after_forced_commits_equals_fresh_prefill():
    _, m = _tiny(D=4)
    prompt = synth.make_prompts(m.cfg, [6], 29)[0]
    forced = synth.make_forced_accepts(40, 1, 4, 3)[:, 0]
    _, rounds, st = om.generate(m, prompt, 20, forced=forced)
    fresh = om.prefill(m, st.tokens[:-1])
    assert fresh.seq_len == st.seq_len
    for li in range(m.cfg.n_layers):
        np.testing.assert_allclose(st.cache_k[li], fresh.cache_k[li], atol=1e-12)
        np.testing.assert_allclose(st.cache_v[li], fresh.cache_v[li], atol=1e-12)
    assert st.seq_len == len(prompt) + sum(n + 1 for n in rounds)
