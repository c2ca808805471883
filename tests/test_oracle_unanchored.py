"""Pins of the oracle's unanchored drafting (the anchored-vs-unanchored ablation).

Reading (the paper does not define the anchor): the unanchored draft's block is
the D masks alone at t+1..t+D; the anchor at position t is cache context
computed as the verifier computes it.  Pinned against the no-cache brute-force
decoder with an explicit per-row adapter flag and visibility matrix, against
plain greedy decoding (the loop stays exact), and against a fresh prefill of the
committed tokens (the cache bookkeeping); planted mistakes fail those pins.
"""
import numpy as np
import pytest

import synth
from oracle import brute
from oracle import model as om

TOL = 1e-9


def _model(D, seed=0):
    cfg = synth.TINY.with_(block=D)
    w = synth.make_weights(cfg, seed)
    return w, om.OracleModel(w)


def _brute_draft(w, prefix, anchor):
    """Rows t..t+D of [prefix, anchor, mask x D]: prompt and anchor rows causal
    without the adapter; mask rows with the adapter, seeing everything."""
    cfg = w.cfg
    t, D = len(prefix), cfg.block
    toks = list(prefix) + [anchor] + [cfg.mask_id] * D
    vis = brute.causal_mask(t + 1 + D)
    vis[t + 1:, :] = True
    return brute.forward_full(w, toks, [False] * (t + 1) + [True] * D, vis)[t:]


def _brute_verify(w, prefix, anchor, drafts):
    toks = list(prefix) + [anchor] + [int(x) for x in drafts]
    return brute.forward_full(w, toks, [False] * len(toks), brute.causal_mask(len(toks)))[len(prefix):]


def _errs(w, m, st):
    prefix = st.tokens[:-1]
    d, p0, dlg, akv = om.draft_unanchored(m, st)
    p, vlg, k, v = om.verify_unanchored(m, st, akv, d)
    ref_d = _brute_draft(w, prefix, st.anchor)
    ref_v = _brute_verify(w, prefix, st.anchor, d)
    return np.abs(dlg - ref_d).max(), np.abs(vlg - ref_v[1:]).max(), d, p0, p, dlg, ref_v


@pytest.mark.parametrize("D,t", [(1, 3), (4, 7), (16, 9), (16, 40)])
def test_unanchored_passes_match_brute_force(D, t):
    w, m = _model(D)
    prompt = synth.make_prompts(m.cfg, [t], 60 + t)[0]
    st = om.prefill(m, prompt)
    ed, ev, d, p0, p, dlg, ref_v = _errs(w, m, st)
    assert ed < TOL and ev < TOL
    # the anchor row is the verifier's row for position t: p_0 and its logits
    # equal those of the anchored verify of [anchor, drafts]
    np.testing.assert_allclose(dlg[0], ref_v[0], atol=TOL, rtol=0)
    p_anch, vl_anch, _, _ = om.verify(m, st, d)
    assert p0 == p_anch[0] and np.array_equal(p, p_anch[1:])
    np.testing.assert_allclose(vl_anch[1:], _brute_verify(w, st.tokens[:-1], st.anchor, d)[1:], atol=TOL, rtol=0)


def test_unanchored_draft_differs_from_anchored():
    """The ablation is not vacuous: without the anchor in the block (adapter
    on, bidirectional) the mask rows' logits change."""
    w, m = _model(16)
    prompt = synth.make_prompts(m.cfg, [20], 12)[0]
    st = om.prefill(m, prompt)
    _, l_anch = om.draft(m, st)
    _, _, l_un, _ = om.draft_unanchored(m, st)
    assert np.abs(l_un[1:] - l_anch[1:]).max() > 1e-3


@pytest.mark.parametrize("forced", [None, [3, 0, 4, 4, 1]])
def test_unanchored_loop_is_greedy_decoding_and_cache_matches_prefill(forced):
    w, m = _model(4)
    prompt = synth.make_prompts(m.cfg, [6], 3)[0]
    st = om.prefill(m, prompt)
    rounds = 5
    for r in range(rounds):
        om.step_unanchored(m, st, None if forced is None else forced[r])
    if forced is None:        # real acceptance keeps the output exact; forced counts do not
        assert st.generated == brute.greedy_decode(w, prompt, len(st.generated))
    # the cache holds every committed token but the anchor, as a fresh prefill would
    fresh = om.prefill(m, st.tokens[:-1])
    for li in range(m.cfg.n_layers):
        np.testing.assert_allclose(st.cache_k[li], fresh.cache_k[li], atol=TOL, rtol=0)
        np.testing.assert_allclose(st.cache_v[li], fresh.cache_v[li], atol=TOL, rtol=0)
    assert fresh.anchor == st.anchor


def _setup():
    w, m = _model(4)
    prompt = synth.make_prompts(m.cfg, [8], 77)[0]
    return w, m, om.prefill(m, prompt)


def test_unplanted_unanchored_matches():
    w, m, st = _setup()
    ed, ev = _errs(w, m, st)[:2]
    assert ed < TOL and ev < TOL


def test_anchor_row_with_adapter_is_caught(monkeypatch):
    w, m, st = _setup()
    real = m.forward_block

    def bad(tokens, pos0, ck, cv, causal, adapter_on, **kw):
        if len(tokens) == 1:
            adapter_on = True
        return real(tokens, pos0, ck, cv, causal, adapter_on, **kw)
    monkeypatch.setattr(m, "forward_block", bad)
    assert _errs(w, m, st)[0] > 1e-6


def test_masks_not_seeing_the_anchor_is_caught(monkeypatch):
    w, m, st = _setup()
    real = m.forward_block

    def bad(tokens, pos0, ck, cv, causal, adapter_on, **kw):
        if len(tokens) > 1 and adapter_on:       # the mask block right after the prefix, no anchor
            ck = [a[:-1] for a in ck]
            cv = [a[:-1] for a in cv]
            pos0 -= 1
        return real(tokens, pos0, ck, cv, causal, adapter_on, **kw)
    monkeypatch.setattr(m, "forward_block", bad)
    assert _errs(w, m, st)[0] > 1e-6


def test_verify_without_the_cached_anchor_is_caught(monkeypatch):
    w, m, st = _setup()
    real = m.forward_block

    def bad(tokens, pos0, ck, cv, causal, adapter_on, **kw):
        if len(tokens) > 1 and not adapter_on:   # the verify of the drafts, anchor dropped
            ck = [a[:-1] for a in ck]
            cv = [a[:-1] for a in cv]
            pos0 -= 1
        return real(tokens, pos0, ck, cv, causal, adapter_on, **kw)
    monkeypatch.setattr(m, "forward_block", bad)
    assert _errs(w, m, st)[1] > 1e-6
