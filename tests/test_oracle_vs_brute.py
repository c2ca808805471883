"""Cached oracle vs the no-cache brute-force decoder (tiny model, float64).

Pins the block bookkeeping of the oracle: positions, prefix/block visibility of
both masks, the per-pass adapter switch, and the commit of accepted rows.
"""
import numpy as np
import pytest

import synth
from oracle import brute
from oracle import model as om

TOL = 1e-9


def _model(D, seed=0, **kw):
    cfg = synth.TINY.with_(block=D, **kw)
    w = synth.make_weights(cfg, seed)
    return w, om.OracleModel(w)


def _check_step(w, m, st, drafts_override=None):
    cfg = m.cfg
    t, W = st.seq_len, cfg.width
    prefix = st.tokens[:-1]
    assert len(prefix) == t
    d_tok, d_lg = om.draft(m, st)
    toks = prefix + [st.anchor] + [cfg.mask_id] * cfg.block
    ref = brute.forward_full(w, toks, [False] * t + [True] * W, brute.draft_mask(t, W))
    np.testing.assert_allclose(d_lg, ref[t:], atol=TOL, rtol=0)
    drafts = d_tok if drafts_override is None else drafts_override
    p, v_lg, k, v = om.verify(m, st, drafts)
    toks = prefix + [st.anchor] + [int(x) for x in drafts]
    ref = brute.forward_full(w, toks, [False] * len(toks), brute.causal_mask(len(toks)))
    np.testing.assert_allclose(v_lg, ref[t:], atol=TOL, rtol=0)
    return drafts, p, k, v


@pytest.mark.parametrize("D,t", [(0, 1), (1, 7), (4, 7), (16, 1), (16, 7), (16, 40)])
def test_draft_and_verify_match_brute_force(D, t):
    w, m = _model(D)
    prompt = synth.make_prompts(m.cfg, [t], 11)[0]
    st = om.prefill(m, prompt)
    _check_step(w, m, st)


def test_prefix_128_matches_brute_force():
    w, m = _model(16)
    prompt = synth.make_prompts(m.cfg, [128], synth.WORKLOADS[0].seed(1))[0]
    st = om.prefill(m, prompt)
    _check_step(w, m, st)


def test_prefill_anchor_is_brute_force_greedy():
    w, m = _model(4)
    prompt = synth.make_prompts(m.cfg, [9], 5)[0]
    st = om.prefill(m, prompt)
    assert st.anchor == brute.greedy_decode(w, prompt, 1)[0]


@pytest.mark.parametrize("forced", [[3, 0, 4], [4, 4, 1]])
def test_multi_step_commit_matches_brute_force(forced):
    """After forced commits, the next draft/verify still match a full recompute."""
    w, m = _model(4)
    prompt = synth.make_prompts(m.cfg, [6], 3)[0]
    st = om.prefill(m, prompt)
    for n in forced:
        drafts, p, k, v = _check_step(w, m, st)
        nn, out = om.accept(drafts, p, forced_n=n)
        om.commit(st, nn, out, k, v)
    _check_step(w, m, st)


def test_qk_norm_off_matches_brute_force():
    w, m = _model(4, qk_norm=False)
    prompt = synth.make_prompts(m.cfg, [5], 2)[0]
    st = om.prefill(m, prompt)
    _check_step(w, m, st)


@pytest.mark.parametrize("k", [1, 2])
def test_early_exit_draft_matches_brute_force(k):
    """The early-exit drafter (first k blocks, then final norm and LM head)
    equals a brute-force pass truncated to the same k blocks."""
    w, m = _model(4)
    prompt = synth.make_prompts(m.cfg, [9], 11)[0]
    st = om.prefill(m, prompt)
    _, d_lg = om.draft(m, st, n_layers=k)
    t, W = len(prompt), m.cfg.width
    toks = list(prompt) + [st.anchor] + [m.cfg.mask_id] * m.cfg.block
    ref = brute.forward_full(w, toks, [False] * t + [True] * W, brute.draft_mask(t, W), n_layers=k)
    np.testing.assert_allclose(d_lg, ref[t:], atol=TOL, rtol=0)


def test_full_depth_early_exit_is_the_draft():
    w, m = _model(16)
    prompt = synth.make_prompts(m.cfg, [20], 12)[0]
    st = om.prefill(m, prompt)
    d0, l0 = om.draft(m, st)
    d1, l1 = om.draft(m, st, n_layers=m.cfg.n_layers)
    assert np.array_equal(d0, d1) and np.array_equal(l0, l1)
    _, l2 = om.draft(m, st, n_layers=1)
    assert np.abs(l2 - l0).max() > 1e-3          # a shallower drafter is a different model
