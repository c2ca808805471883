"""The oracle's pins catch plausible mistakes.

Each case plants one mistake in a copy of the oracle's arithmetic (on the CPU,
via monkeypatch) and checks that a brute-force comparison or an invariant used
to pin the oracle then fails.
"""
import numpy as np
import pytest

import synth
from oracle import brute
from oracle import model as om


def _setup():
    cfg = synth.TINY.with_(block=4)
    w = synth.make_weights(cfg, 0)
    m = om.OracleModel(w)
    prompt = synth.make_prompts(cfg, [6], 31)[0]
    return w, m, prompt


def _draft_err(w, m, prompt):
    st = om.prefill(m, prompt)
    _, lg = om.draft(m, st)
    t, W = len(prompt), m.cfg.width
    toks = list(prompt) + [st.anchor] + [m.cfg.mask_id] * m.cfg.block
    ref = brute.forward_full(w, toks, [False] * t + [True] * W, brute.draft_mask(t, W))
    return np.abs(lg - ref[t:]).max()


def _verify_err(w, m, prompt):
    st = om.prefill(m, prompt)
    drafts = [3, 4, 5, 6]
    _, lg, _, _ = om.verify(m, st, drafts)
    toks = list(prompt) + [st.anchor] + drafts
    ref = brute.forward_full(w, toks, [False] * len(toks), brute.causal_mask(len(toks)))
    return np.abs(lg - ref[len(prompt):]).max()


def test_unplanted_oracle_matches():
    w, m, prompt = _setup()
    assert _draft_err(w, m, prompt) < 1e-9
    assert _verify_err(w, m, prompt) < 1e-9


def test_rope_sign_flip_is_caught(monkeypatch):
    w, m, prompt = _setup()
    real = om.rope
    monkeypatch.setattr(om, "rope", lambda v, p, th: real(v, -p, th))
    assert _verify_err(w, m, prompt) > 1e-6


def test_dropped_lora_scale_is_caught(monkeypatch):
    w, m, prompt = _setup()
    monkeypatch.setattr(m.cfg.__class__, "lora_scale", property(lambda s: 1.0))
    assert _draft_err(w, m, prompt) > 1e-6


def test_transposed_lora_operands_are_caught(monkeypatch):
    w, m, prompt = _setup()

    def bad_linear(layer, name, x, on):
        y = x @ layer[name].T
        if on:
            A, B = layer["lora"][name]
            y = y + m.cfg.lora_scale * ((x @ A.T) @ B[::-1].T)   # rows of B reversed
        return y
    monkeypatch.setattr(m, "linear", bad_linear)
    assert _draft_err(w, m, prompt) > 1e-6


def test_causal_verify_without_mask_is_caught(monkeypatch):
    w, m, prompt = _setup()
    real = om.verify
    monkeypatch.setattr(om, "verify", lambda mm, st, d, adapter_on=False, causal=True:
                        real(mm, st, d, adapter_on, causal=False))
    assert _verify_err(w, m, prompt) > 1e-6


def test_missing_eps_or_gain_is_caught(monkeypatch):
    w, m, prompt = _setup()
    monkeypatch.setattr(om, "rms_norm", lambda x, g, eps: x / np.sqrt(np.mean(x * x, -1, keepdims=True) + eps))
    assert _verify_err(w, m, prompt) > 1e-6


def test_off_by_one_acceptance_is_caught(monkeypatch):
    # planted in the oracle: draft x_i compared with p_i instead of p_{i-1};
    # the hand table of the acceptance rule must then fail
    import test_accept

    def bad_accept(drafts, p, forced_n=None):
        n = 0
        while n < len(drafts) and int(drafts[n]) == int(p[n + 1]):
            n += 1
        return n, [int(t) for t in drafts[:n]] + [int(p[n])]
    monkeypatch.setattr(om, "accept", bad_accept)
    failed = [row for row in test_accept.TABLE if om.accept(row[0], test_accept.P) != (row[1], row[2])]
    assert failed


def test_wrong_kv_head_mapping_is_caught(monkeypatch):
    w, m, prompt = _setup()
    # swap the two KV heads' key projections in the oracle's copy only
    for lw in m.layers:
        d = m.cfg.head_dim
        k = lw["k"].copy()
        lw["k"] = np.concatenate([k[d:], k[:d]], axis=0)
    assert _verify_err(w, m, prompt) > 1e-6
