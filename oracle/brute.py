"""Brute-force reference decoder (test infrastructure only).

No KV cache, no block bookkeeping: every call recomputes all positions of a
token sequence from scratch, row by row, with an explicit visibility matrix
and a per-row adapter flag.  It shares no helper with ``oracle.model`` so that
the cached oracle can be checked against it on tiny inputs:

* a PEFT-BD draft at state (prompt of length t, anchor) equals the rows t..t+D
  of a full pass over prompt + [anchor, mask x D] where prompt rows are
  adapter-off and causal, and block rows are adapter-on and see the prompt and
  every block row (Sec. 3 steps 1-2, App. A.4);
* a verify equals the same full pass with the drafts in place of the masks,
  adapter off everywhere, causal everywhere (Sec. 3 step 3);
* greedy decoding is repeated argmax of the last row of a causal full pass,
  the reference for the exact greedy audit (App. A.1, Tab. HF diagnostics).
"""
from __future__ import annotations

import math
from typing import List, Sequence

import numpy as np

from synth import Weights


def _norm_row(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    acc = 0.0
    for val in x:
        acc += float(val) * float(val)
    return x * (1.0 / math.sqrt(acc / len(x) + eps)) * g


def _rotate(vec: np.ndarray, pos: int, theta: float) -> np.ndarray:
    d = len(vec)
    half = d // 2
    out = np.empty(d)
    for i in range(half):
        ang = pos * theta ** (-2.0 * i / d)
        c, s = math.cos(ang), math.sin(ang)
        out[i] = vec[i] * c - vec[i + half] * s
        out[i + half] = vec[i + half] * c + vec[i] * s
    return out


def forward_full(w: Weights, tokens: Sequence[int], adapter_rows: Sequence[bool],
                 visible: np.ndarray, n_layers=None) -> np.ndarray:
    """Logits [n, V] of a full no-cache pass; visible[i, j]: row i sees key j.
    n_layers: only the first n_layers blocks before the final norm (None: all)."""
    cfg = w.cfg
    n = len(tokens)
    d, hq, hkv = cfg.head_dim, cfg.n_q_heads, cfg.n_kv_heads
    f = lambda a: np.asarray(a, dtype=np.float64)
    s_lora = cfg.lora_alpha / cfg.lora_rank
    x = np.stack([f(w.embed[t]) for t in tokens])

    def proj(lw, name, row_vec, on):
        y = f(getattr(lw, name)) @ row_vec
        if on:
            A, B = lw.lora[name]
            y = y + s_lora * (f(B) @ (f(A) @ row_vec))
        return y

    for lw in w.layers[:n_layers]:
        Q = np.zeros((n, hq, d)); K = np.zeros((n, hkv, d)); Vv = np.zeros((n, hkv, d))
        for i in range(n):
            xn = _norm_row(x[i], f(lw.attn_norm), cfg.rms_eps)
            qi = proj(lw, "q", xn, adapter_rows[i]).reshape(hq, d)
            ki = proj(lw, "k", xn, adapter_rows[i]).reshape(hkv, d)
            vi = proj(lw, "v", xn, adapter_rows[i]).reshape(hkv, d)
            for h in range(hq):
                qh = _norm_row(qi[h], f(lw.q_norm), cfg.rms_eps) if cfg.qk_norm else qi[h]
                Q[i, h] = _rotate(qh, i, cfg.rope_theta)
            for h in range(hkv):
                kh = _norm_row(ki[h], f(lw.k_norm), cfg.rms_eps) if cfg.qk_norm else ki[h]
                K[i, h] = _rotate(kh, i, cfg.rope_theta)
                Vv[i, h] = vi[h]
        x_new = np.empty_like(x)
        for i in range(n):
            att = np.zeros(hq * d)
            for h in range(hq):
                g = (h * hkv) // hq
                keys = [j for j in range(n) if visible[i, j]]
                sc = np.array([float(Q[i, h] @ K[j, g]) / math.sqrt(d) for j in keys])
                wts = np.exp(sc - sc.max())
                wts = wts / wts.sum()
                att[h * d:(h + 1) * d] = sum(wt * Vv[j, g] for wt, j in zip(wts, keys))
            xi = x[i] + proj(lw, "o", att, adapter_rows[i])
            xm = _norm_row(xi, f(lw.mlp_norm), cfg.rms_eps)
            gt = proj(lw, "gate", xm, adapter_rows[i])
            up = proj(lw, "up", xm, adapter_rows[i])
            hmid = gt / (1.0 + np.exp(-gt)) * up
            x_new[i] = xi + proj(lw, "down", hmid, adapter_rows[i])
        x = x_new
    E = f(w.embed)
    out = np.empty((n, cfg.vocab))
    for i in range(n):
        out[i] = E @ _norm_row(x[i], f(w.final_norm), cfg.rms_eps)
    return out


def causal_mask(n: int) -> np.ndarray:
    return np.tril(np.ones((n, n), dtype=bool))


def draft_mask(t: int, width: int) -> np.ndarray:
    """Prompt rows causal; block rows see the prompt and the whole block."""
    n = t + width
    m = causal_mask(n)
    m[t:, :] = True
    return m


def greedy_decode(w: Weights, prompt: Sequence[int], n_new: int) -> List[int]:
    """Plain greedy decoding by full recomputation (lowest id wins ties)."""
    seq = list(prompt)
    out = []
    for _ in range(n_new):
        lg = forward_full(w, seq, [False] * len(seq), causal_mask(len(seq)))
        nxt = int(np.argmax(lg[-1]))
        out.append(nxt)
        seq.append(nxt)
    return out
