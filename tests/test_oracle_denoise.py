"""Pins of the oracle's multi-step denoising (the denoising-steps ablation).

The paper states the ablation (one vs two draft passes per step) but no
remasking rule; the oracle's reading is low-confidence remasking: pass s fixes
the n_s still-masked positions whose candidate has the highest log-probability,
with D split over the passes as evenly as possible (larger shares first).

What pins it:
* the schedule against its closed form and hand values;
* the confidence against scipy's log-softmax and hand-computed rows;
* the selection against an exhaustive search for the one subset that
  dominates its complement;
* the whole k-pass procedure against a brute-force run of the same procedure
  built on the no-cache full-sequence forward, scipy's log-softmax and the
  exhaustive selection;
* k = 1 against the one-step draft (identical), and planted mistakes.
"""
import itertools
import math

import numpy as np
import pytest
from scipy.special import log_softmax

import synth
from oracle import brute
from oracle import model as om

TOL = 1e-9


def _model(D, seed=0):
    cfg = synth.TINY.with_(block=D)
    w = synth.make_weights(cfg, seed)
    return w, om.OracleModel(w)


# -- schedule ----------------------------------------------------------------

def test_schedule_closed_form():
    for D in range(1, 33):
        for k in range(1, D + 1):
            s = om.denoise_schedule(D, k)
            assert len(s) == k and sum(s) == D
            assert all(a >= b for a, b in zip(s, s[1:]))
            assert max(s) - min(s) <= 1 and min(s) >= 1
    assert om.denoise_schedule(16, 1) == [16]
    assert om.denoise_schedule(16, 2) == [8, 8]
    assert om.denoise_schedule(16, 3) == [6, 5, 5]
    assert om.denoise_schedule(16, 16) == [1] * 16
    assert om.denoise_schedule(32, 5) == [7, 7, 6, 6, 6]
    for bad in (0, 17):
        with pytest.raises(ValueError):
            om.denoise_schedule(16, bad)


# -- confidence ----------------------------------------------------------------

def test_confidence_hand_values():
    # mask id 2 holds the largest logit: the candidate is id 1, p = 3 / 8
    tok, c = om.candidate_confidence(np.log(np.array([1.0, 3.0, 4.0])), mask_id=2)
    assert tok == 1 and abs(c - math.log(3 / 8)) < 1e-15
    # tie between ids 0 and 1: the lower id; p = e / (2e + 1)
    tok, c = om.candidate_confidence(np.array([1.0, 1.0, 0.0]), mask_id=2)
    assert tok == 0 and abs(c - (1.0 - math.log(2 * math.e + 1))) < 1e-15
    # a constant row over V ids: p = 1 / V
    tok, c = om.candidate_confidence(np.full(64, 7.5), mask_id=63)
    assert tok == 0 and abs(c + math.log(64)) < 1e-14


def test_confidence_matches_scipy_log_softmax():
    rng = np.random.default_rng(5)
    for _ in range(20):
        V = int(rng.integers(2, 300))
        row = rng.normal(0, 6, V)
        mask = int(rng.integers(0, V))
        tok, c = om.candidate_confidence(row, mask)
        ref = log_softmax(row)
        alt = row.copy()
        alt[mask] = -np.inf
        assert tok == int(np.argmax(alt)) and abs(c - ref[tok]) < 1e-12


# -- selection -----------------------------------------------------------------

def _dominant_subset(conf: dict, n: int):
    """Exhaustive: the one n-subset every member of which beats every
    non-member (higher confidence, or equal confidence and lower position)."""
    keys = sorted(conf)
    beats = lambda i, j: conf[i] > conf[j] or (conf[i] == conf[j] and i < j)
    found = [list(S) for S in itertools.combinations(keys, n)
             if all(beats(i, j) for i in S for j in keys if j not in S)]
    assert len(found) == 1
    return found[0]


def test_selection_is_the_dominant_subset():
    rng = np.random.default_rng(9)
    for _ in range(200):
        D = int(rng.integers(1, 9))
        masked = sorted(rng.choice(D, size=int(rng.integers(1, D + 1)), replace=False).tolist())
        conf = {j: float(np.round(rng.normal(), 1)) for j in masked}     # rounding makes ties
        n = int(rng.integers(1, len(masked) + 1))
        assert om.remask_select(conf, n) == _dominant_subset(conf, n)


# -- the k-pass procedure --------------------------------------------------------

def _brute_denoise(w, prompt, anchor, n_steps):
    """The same procedure on the no-cache full-sequence forward."""
    cfg = w.cfg
    D, mask, t, W = cfg.block, cfg.mask_id, len(prompt), cfg.width
    block = [mask] * D
    conf = np.full(D, np.nan)
    fixed_at = np.zeros(D, dtype=np.int32)
    lg = None
    for s, n_s in enumerate(om.denoise_schedule(D, n_steps), start=1):
        toks = list(prompt) + [anchor] + block
        lg = brute.forward_full(w, toks, [False] * t + [True] * W, brute.draft_mask(t, W))[t:]
        cand = {}
        for j in range(D):
            if fixed_at[j]:
                continue
            row = lg[j + 1].copy()
            row[mask] = -np.inf
            tok = int(np.argmax(row))
            cand[j] = (tok, float(log_softmax(lg[j + 1])[tok]))
        for j in _dominant_subset({j: c for j, (_, c) in cand.items()}, n_s):
            block[j], conf[j], fixed_at[j] = cand[j][0], cand[j][1], s
    return np.array(block), lg, conf, fixed_at


@pytest.mark.parametrize("D,k,t", [(4, 2, 7), (4, 3, 7), (4, 4, 1), (6, 4, 12), (16, 2, 9)])
def test_denoise_matches_brute_force(D, k, t):
    w, m = _model(D)
    prompt = synth.make_prompts(m.cfg, [t], 40 + t)[0]
    st = om.prefill(m, prompt)
    tok, lg, conf, fixed_at = om.draft_denoise(m, st, k)
    rtok, rlg, rconf, rfixed = _brute_denoise(w, prompt, st.anchor, k)
    assert np.array_equal(tok, rtok) and np.array_equal(fixed_at, rfixed)
    np.testing.assert_allclose(conf, rconf, atol=TOL, rtol=0)
    np.testing.assert_allclose(lg, rlg, atol=TOL, rtol=0)
    # every position fixed exactly once, in the scheduled numbers, never the mask id
    sched = om.denoise_schedule(D, k)
    assert [int((fixed_at == s).sum()) for s in range(1, k + 1)] == sched
    assert not np.any(tok == m.cfg.mask_id)


def test_one_pass_is_the_one_step_draft():
    w, m = _model(16)
    prompt = synth.make_prompts(m.cfg, [20], 12)[0]
    st = om.prefill(m, prompt)
    d0, l0 = om.draft(m, st)
    d1, l1, conf, fixed_at = om.draft_denoise(m, st, 1)
    assert np.array_equal(d0, d1) and np.array_equal(l0, l1)
    assert np.all(fixed_at == 1)
    ref = log_softmax(l0[1:], axis=-1)[np.arange(16), d0]
    np.testing.assert_allclose(conf, ref, atol=1e-12, rtol=0)


def test_later_passes_see_the_fixed_tokens():
    """The last pass runs over a block holding the earlier passes' tokens, so
    its logits differ from the one-step draft's."""
    w, m = _model(16)
    prompt = synth.make_prompts(m.cfg, [20], 12)[0]
    st = om.prefill(m, prompt)
    _, l0 = om.draft(m, st)
    _, l2, _, fixed_at = om.draft_denoise(m, st, 2)
    assert sorted(np.bincount(fixed_at)[1:].tolist()) == [8, 8]
    assert np.abs(l2 - l0).max() > 1e-3


# -- planted mistakes -------------------------------------------------------------

def _denoise_vs_brute(w, m, prompt, k=3):
    st = om.prefill(m, prompt)
    tok, lg, conf, fixed_at = om.draft_denoise(m, st, k)
    rtok, rlg, rconf, rfixed = _brute_denoise(w, prompt, st.anchor, k)
    return (np.array_equal(tok, rtok) and np.array_equal(fixed_at, rfixed)
            and np.abs(conf - rconf).max() < TOL and np.abs(lg - rlg).max() < TOL)


def _setup():
    w, m = _model(6)
    return w, m, synth.make_prompts(m.cfg, [8], 77)[0]


def test_unplanted_denoise_matches():
    assert _denoise_vs_brute(*_setup())


def test_lowest_confidence_first_is_caught(monkeypatch):
    w, m, prompt = _setup()
    real = om.remask_select
    monkeypatch.setattr(om, "remask_select", lambda c, n: real({j: -v for j, v in c.items()}, n))
    assert not _denoise_vs_brute(w, m, prompt)


def test_max_logit_confidence_is_caught(monkeypatch):
    w, m, prompt = _setup()

    def bad(row, mask_id):
        tok = om.greedy_argmax(row, exclude=mask_id)
        return tok, float(row[tok])                 # unnormalised logit
    monkeypatch.setattr(om, "candidate_confidence", bad)
    assert not _denoise_vs_brute(w, m, prompt)


def test_mask_left_out_of_the_normaliser_is_caught(monkeypatch):
    w, m, prompt = _setup()

    def bad(row, mask_id):
        r = np.delete(row, mask_id)
        tok = om.greedy_argmax(row, exclude=mask_id)
        mx = r.max()
        return tok, float(row[tok] - mx - np.log(np.exp(r - mx).sum()))
    monkeypatch.setattr(om, "candidate_confidence", bad)
    assert not _denoise_vs_brute(w, m, prompt)


def test_block_tokens_ignored_is_caught(monkeypatch):
    w, m, prompt = _setup()
    real = om.draft_block_logits
    monkeypatch.setattr(om, "draft_block_logits",
                        lambda mm, st, block, a=True, c=False: real(mm, st, [mm.cfg.mask_id] * len(block), a, c))
    assert not _denoise_vs_brute(w, m, prompt)
