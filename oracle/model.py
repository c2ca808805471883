"""CPU oracle of one PEFT-BD speculative step (test infrastructure only).

Only the tests, the package's smoke check and the benchmark's CPU-baseline leg
use this module; the product path never imports it.  It is plain NumPy in
float64 and follows the paper's statement of the method:

* Sec. 3 (enumerated algorithm): with the adapter on, append D masked
  positions and denoise the block in one step (draft); with the adapter off,
  run the autoregressive verifier on the proposed block; accept the longest
  matching prefix; append and repeat.
* App. A.1: verification is exact greedy top-1 matching; the longest matching
  prefix is accepted.
* App. A.2: the adapter is LoRA on every linear projection of every block,
  y = W x + (alpha/r) B (A x), backbone frozen.
* App. A.4: both passes have token width 17 = D + 1; the adapter is on for the
  whole draft pass and off for the whole verify pass; the draft pass keeps
  its block K/V as scratch only, and the verify pass uses a different (causal)
  attention mask.

Readings where the paper is silent (the model architecture is Qwen3-0.6B's
public definition, which the paper does not print):
  * block row 0 is the anchor: the last committed token, not yet in the KV
    cache; draft token j (j = 1..D) is the argmax of block row j (the masked
    position's own prediction); the draft argmax excludes the mask id;
  * draft rows see the whole committed prefix and every block row; verify rows
    see the prefix and the block rows up to their own (causal);
  * the prefix K/V is the adapter-off cache; the draft never writes the cache;
  * after accepting n drafts the n+1 tokens x1..xn, p_n are committed, the
    cache keeps rows t..t+n and the new anchor is the bonus token p_n;
  * argmax ties go to the lowest token id.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional, Sequence

import numpy as np

from synth import LORA_TARGETS, ModelConfig, Weights


# ---------------------------------------------------------------------------
# Elementary operations
# ---------------------------------------------------------------------------

def rms_norm(x: np.ndarray, gain: np.ndarray, eps: float) -> np.ndarray:
    """RMSNorm over the last axis: x / sqrt(mean(x^2) + eps) * gain."""
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * gain


def rope(v: np.ndarray, positions: np.ndarray, theta: float) -> np.ndarray:
    """Rotary embedding, rotate-half pairing (i, i + d/2).

    v: [n, heads, d]; positions: [n].  Frequency of pair i is theta^(-2i/d).
    """
    d = v.shape[-1]
    half = d // 2
    inv_freq = theta ** (-(np.arange(half, dtype=np.float64) * 2.0) / d)
    ang = positions.astype(np.float64)[:, None] * inv_freq[None, :]   # [n, half]
    cos = np.cos(ang)[:, None, :]
    sin = np.sin(ang)[:, None, :]
    a = v[..., :half]
    b = v[..., half:]
    return np.concatenate([a * cos - b * sin, b * cos + a * sin], axis=-1).astype(v.dtype, copy=False)


def silu(x: np.ndarray) -> np.ndarray:
    return x / (1.0 + np.exp(-x))


def softmax_rows(s: np.ndarray) -> np.ndarray:
    m = np.max(s, axis=-1, keepdims=True)
    e = np.exp(s - m)
    return e / np.sum(e, axis=-1, keepdims=True)


def greedy_argmax(logits: np.ndarray, exclude: Optional[int] = None) -> int:
    """Top-1 token id; ties go to the lowest id (np.argmax keeps the first)."""
    if exclude is not None:
        logits = logits.copy()
        logits[exclude] = -np.inf
    return int(np.argmax(logits))


# ---------------------------------------------------------------------------
# Model
# ---------------------------------------------------------------------------

class OracleModel:
    """The backbone plus its LoRA adapter, held in float64 (the benchmark's
    host baseline also runs it with float32 arrays; parity uses float64)."""

    def __init__(self, w: Weights, dtype=np.float64):
        f = lambda a: np.asarray(a, dtype=dtype)
        self.cfg: ModelConfig = w.cfg
        self.embed = f(w.embed)
        self.final_norm = f(w.final_norm)
        self.layers = []
        for lw in w.layers:
            self.layers.append(dict(
                attn_norm=f(lw.attn_norm), mlp_norm=f(lw.mlp_norm),
                q_norm=f(lw.q_norm), k_norm=f(lw.k_norm),
                q=f(lw.q), k=f(lw.k), v=f(lw.v), o=f(lw.o),
                gate=f(lw.gate), up=f(lw.up), down=f(lw.down),
                lora={n: (f(lw.lora[n][0]), f(lw.lora[n][1])) for n in LORA_TARGETS},
            ))

    # App. A.2: y = W x + (alpha / r) * B (A x) when the adapter is enabled.
    def linear(self, layer: dict, name: str, x: np.ndarray, adapter_on: bool) -> np.ndarray:
        y = x @ layer[name].T
        if adapter_on:
            A, B = layer["lora"][name]
            y = y + self.cfg.lora_scale * ((x @ A.T) @ B.T)
        return y

    def logits(self, x: np.ndarray) -> np.ndarray:
        """Final RMSNorm and the tied LM head (embedding matrix)."""
        return rms_norm(x, self.final_norm, self.cfg.rms_eps) @ self.embed.T

    def forward_block(self, tokens: Sequence[int], pos0: int,
                      cache_k: List[np.ndarray], cache_v: List[np.ndarray],
                      causal: bool, adapter_on: bool,
                      logit_rows: Optional[Sequence[int]] = None,
                      n_layers: Optional[int] = None):
        """Run n block rows at positions pos0..pos0+n-1 over a committed prefix.

        cache_k[l], cache_v[l]: [pos0, h_kv, d] post-norm post-RoPE keys and
        values of the committed prefix (all visible to every block row).  Block
        key i is visible to block row j iff (not causal) or i <= j.
        n_layers: run only the first n_layers blocks before the final norm and
        the LM head (an early-exit drafter; None = all).
        Returns (logits [len(logit_rows), V], new_k [L][n,h_kv,d], new_v).
        """
        cfg = self.cfg
        n = len(tokens)
        d, hq, hkv = cfg.head_dim, cfg.n_q_heads, cfg.n_kv_heads
        group = hq // hkv
        positions = pos0 + np.arange(n)
        x = self.embed[np.asarray(tokens, dtype=np.int64)]
        block_vis = np.tril(np.ones((n, n), dtype=bool)) if causal else np.ones((n, n), dtype=bool)
        new_k, new_v = [], []
        for li, lw in enumerate(self.layers[:n_layers]):
            xn = rms_norm(x, lw["attn_norm"], cfg.rms_eps)
            q = self.linear(lw, "q", xn, adapter_on).reshape(n, hq, d)
            k = self.linear(lw, "k", xn, adapter_on).reshape(n, hkv, d)
            v = self.linear(lw, "v", xn, adapter_on).reshape(n, hkv, d)
            if cfg.qk_norm:
                q = rms_norm(q, lw["q_norm"], cfg.rms_eps)
                k = rms_norm(k, lw["k_norm"], cfg.rms_eps)
            q = rope(q, positions, cfg.rope_theta)
            k = rope(k, positions, cfg.rope_theta)
            new_k.append(k)
            new_v.append(v)
            K = np.concatenate([cache_k[li], k], axis=0)          # [pos0+n, hkv, d]
            V = np.concatenate([cache_v[li], v], axis=0)
            vis = np.concatenate([np.ones((n, pos0), dtype=bool), block_vis], axis=1)
            o = np.empty((n, hq, d), dtype=x.dtype)
            for h in range(hq):
                g = h // group
                s = (q[:, h, :] @ K[:, g, :].T) / np.sqrt(d)       # [n, pos0+n]
                s = np.where(vis, s, -np.inf)
                o[:, h, :] = softmax_rows(s) @ V[:, g, :]
            x = x + self.linear(lw, "o", o.reshape(n, hq * d), adapter_on)
            xm = rms_norm(x, lw["mlp_norm"], cfg.rms_eps)
            hmid = silu(self.linear(lw, "gate", xm, adapter_on)) * self.linear(lw, "up", xm, adapter_on)
            x = x + self.linear(lw, "down", hmid, adapter_on)
        rows = range(n) if logit_rows is None else logit_rows
        lg = self.logits(x[list(rows)])
        return lg, new_k, new_v


# ---------------------------------------------------------------------------
# The speculative step
# ---------------------------------------------------------------------------

@dataclass
class SeqState:
    """Committed state of one sequence: adapter-off KV of positions [0, t)."""
    cache_k: List[np.ndarray]     # per layer [t, h_kv, d]
    cache_v: List[np.ndarray]
    anchor: int                   # last committed token, not yet in the cache
    tokens: List[int] = field(default_factory=list)   # all committed tokens
    generated: List[int] = field(default_factory=list)

    @property
    def seq_len(self) -> int:
        return self.cache_k[0].shape[0]


def prefill(model: OracleModel, prompt: Sequence[int]) -> SeqState:
    """Adapter-off causal pass over the prompt; its greedy next token is the
    first generated token and the first anchor."""
    cfg = model.cfg
    empty = [np.zeros((0, cfg.n_kv_heads, cfg.head_dim), dtype=model.embed.dtype) for _ in range(cfg.n_layers)]
    lg, k, v = model.forward_block(prompt, 0, empty, empty, causal=True,
                                   adapter_on=False, logit_rows=[len(prompt) - 1])
    anchor = greedy_argmax(lg[0])
    return SeqState(k, v, anchor, tokens=list(prompt) + [anchor], generated=[anchor])


def draft(model: OracleModel, st: SeqState, adapter_on: bool = True, causal: bool = False,
          n_layers: Optional[int] = None):
    """Draft pass (Sec. 3 steps 1-2): block [anchor, mask x D] at positions
    t..t+D, adapter on, bidirectional inside the block.  Returns the D draft
    tokens (argmax of rows 1..D over v != mask id) and the logits of all
    D+1 rows.  The cache is not modified (the block K/V is scratch).
    n_layers < L gives the early-exit drafter whose cost the draft-cost
    analysis (App. A.7) varies: the first n_layers blocks, then the final norm
    and the LM head."""
    cfg = model.cfg
    tokens = [st.anchor] + [cfg.mask_id] * cfg.block
    lg, _, _ = model.forward_block(tokens, st.seq_len, st.cache_k, st.cache_v,
                                   causal=causal, adapter_on=adapter_on, n_layers=n_layers)
    drafts = [greedy_argmax(lg[j], exclude=cfg.mask_id) for j in range(1, cfg.block + 1)]
    return np.array(drafts, dtype=np.int32), lg


# ---------------------------------------------------------------------------
# Multi-step denoising: the one- vs two-step ablation (Sec. 4.4, Sec. 5.3;
# the Limitations note that the adapter was trained for one step only).
#
# The paper names the ablation but not its remasking rule.  Readings:
#  * k draft passes; pass s fixes n_s positions, D split as evenly as
#    possible with the larger shares first;
#  * every pass runs the draft pass of Sec. 3 over the current block
#    [anchor, y_1..y_D], where y_j is the token fixed at an earlier pass or the
#    mask id;
#  * the candidate of a still-masked position j is the argmax of row j over
#    v != mask id (as in the one-step draft), and its confidence is the
#    log-probability of that candidate under the softmax of the whole row
#    (all V ids);
#  * the n_s still-masked positions of highest confidence are fixed (equal
#    confidences: lower position first); the others are re-masked, and a fixed
#    position never changes again.
# With k = 1 this is the one-step draft.
# ---------------------------------------------------------------------------

def denoise_schedule(D: int, n_steps: int) -> List[int]:
    """Number of positions fixed at each of the n_steps passes (1 <= n_steps <= D)."""
    if not 1 <= n_steps <= D:
        raise ValueError("n_steps must lie in [1, D]")
    base, rem = divmod(D, n_steps)
    return [base + (1 if s < rem else 0) for s in range(n_steps)]


def draft_block_logits(model: OracleModel, st: SeqState, block: Sequence[int],
                       adapter_on: bool = True, causal: bool = False) -> np.ndarray:
    """Draft pass over a partly denoised block [anchor, y_1..y_D] at positions
    t..t+D (adapter on, bidirectional inside the block); the logits of all
    D+1 rows.  The cache is not modified."""
    tokens = [st.anchor] + [int(t) for t in block]
    lg, _, _ = model.forward_block(tokens, st.seq_len, st.cache_k, st.cache_v,
                                   causal=causal, adapter_on=adapter_on)
    return lg


def candidate_confidence(row: np.ndarray, mask_id: int):
    """(candidate, confidence) of one masked row: the argmax over v != mask id
    and its log-probability under the softmax of the whole row."""
    tok = greedy_argmax(row, exclude=mask_id)
    mx = float(np.max(row))
    lse = mx + float(np.log(np.sum(np.exp(row - mx))))
    return tok, float(row[tok]) - lse


def remask_select(conf: dict, n: int) -> List[int]:
    """The n positions of highest confidence among conf's keys (the still-masked
    positions); equal confidences go to the lower position."""
    order = sorted(conf, key=lambda j: (-conf[j], j))
    return sorted(order[:n])


def draft_denoise(model: OracleModel, st: SeqState, n_steps: int,
                  adapter_on: bool = True, causal: bool = False):
    """k-step draft.  Returns the D draft tokens, the logits of the last pass,
    the confidence at which each position was fixed and the pass (1..k) that
    fixed it."""
    cfg = model.cfg
    D, mask = cfg.block, cfg.mask_id
    block = [mask] * D
    conf = np.full(D, np.nan)
    fixed_at = np.zeros(D, dtype=np.int32)
    lg = None
    for s, n_s in enumerate(denoise_schedule(D, n_steps), start=1):
        lg = draft_block_logits(model, st, block, adapter_on, causal)
        cand = {j: candidate_confidence(lg[j + 1], mask) for j in range(D) if fixed_at[j] == 0}
        for j in remask_select({j: c for j, (_, c) in cand.items()}, n_s):
            block[j], conf[j], fixed_at[j] = cand[j][0], cand[j][1], s
    return np.array(block, dtype=np.int32), lg, conf, fixed_at


def verify(model: OracleModel, st: SeqState, drafts: Sequence[int],
           adapter_on: bool = False, causal: bool = True):
    """Verify pass (Sec. 3 step 3): block [anchor, x1..xD], adapter off,
    causal.  Returns the verifier's greedy tokens p_0..p_D, the logits and the
    block K/V (to be committed at positions t..t+D)."""
    tokens = [st.anchor] + [int(t) for t in drafts]
    lg, k, v = model.forward_block(tokens, st.seq_len, st.cache_k, st.cache_v,
                                   causal=causal, adapter_on=adapter_on)
    p = np.array([greedy_argmax(lg[j]) for j in range(len(tokens))], dtype=np.int32)
    return p, lg, k, v


# ---------------------------------------------------------------------------
# Unanchored drafting: the anchored-vs-unanchored ablation (Sec. 4.4, Sec. 5.3).
#
# The paper does not define the anchor.  Reading: the anchored draft puts the
# anchor (the last committed token, position t) into the block, with the
# adapter on, attending bidirectionally with the masks; the unanchored draft's
# block is the D masks alone at t+1..t+D, and the anchor is context already in
# the cache, computed as the verifier computes it (adapter off, seeing the
# prefix and itself).  The anchor's verifier row also yields p_0, so the
# verify that follows covers the D drafts alone; together they give the same
# K/V and predictions p_0..p_D as the anchored verify of [anchor, drafts].
# ---------------------------------------------------------------------------

def draft_unanchored(model: OracleModel, st: SeqState, adapter_on: bool = True, causal: bool = False):
    """Unanchored draft.  Returns the D draft tokens, p_0 (the verifier's
    prediction after the anchor), the logits of the anchor row and the D mask
    rows ([D+1, V]) and the anchor's K/V (per layer [1, h_kv, d])."""
    cfg = model.cfg
    lg0, k0, v0 = model.forward_block([st.anchor], st.seq_len, st.cache_k, st.cache_v,
                                      causal=True, adapter_on=False)
    ck = [np.concatenate([a, b], axis=0) for a, b in zip(st.cache_k, k0)]
    cv = [np.concatenate([a, b], axis=0) for a, b in zip(st.cache_v, v0)]
    lg, _, _ = model.forward_block([cfg.mask_id] * cfg.block, st.seq_len + 1, ck, cv,
                                   causal=causal, adapter_on=adapter_on)
    drafts = [greedy_argmax(lg[j], exclude=cfg.mask_id) for j in range(cfg.block)]
    return (np.array(drafts, dtype=np.int32), greedy_argmax(lg0[0]),
            np.concatenate([lg0, lg], axis=0), (k0, v0))


def verify_unanchored(model: OracleModel, st: SeqState, anchor_kv, drafts: Sequence[int],
                      adapter_on: bool = False, causal: bool = True):
    """Verify of the D drafts alone at t+1..t+D over the prefix plus the
    anchor's K/V.  Returns p_1..p_D, their logits ([D, V]) and the K/V of rows
    t..t+D (the anchor's first) to be committed."""
    k0, v0 = anchor_kv
    ck = [np.concatenate([a, b], axis=0) for a, b in zip(st.cache_k, k0)]
    cv = [np.concatenate([a, b], axis=0) for a, b in zip(st.cache_v, v0)]
    lg, k, v = model.forward_block([int(t) for t in drafts], st.seq_len + 1, ck, cv,
                                   causal=causal, adapter_on=adapter_on)
    p = np.array([greedy_argmax(lg[j]) for j in range(len(drafts))], dtype=np.int32)
    kk = [np.concatenate([a, b], axis=0) for a, b in zip(k0, k)]
    vv = [np.concatenate([a, b], axis=0) for a, b in zip(v0, v)]
    return p, lg, kk, vv


def step_unanchored(model: OracleModel, st: SeqState, forced_n: Optional[int] = None):
    """One unanchored speculative step: draft, verify, accept, commit."""
    drafts, p0, dlg, akv = draft_unanchored(model, st)
    p_rest, vlg, k, v = verify_unanchored(model, st, akv, drafts)
    p = np.concatenate([[p0], p_rest]).astype(np.int32)
    n, out = accept(drafts, p, forced_n)
    commit(st, n, out, k, v)
    return dict(drafts=drafts, draft_logits=dlg, p=p, verify_logits=vlg, n=n, out=out)


def accept(drafts: Sequence[int], p: Sequence[int], forced_n: Optional[int] = None):
    """Longest-prefix acceptance (Sec. 3 step 4, App. A.1).

    n = largest k <= D with drafts[i-1] == p[i-1] for every i <= k (draft x_i
    is compared with the verifier's prediction for the same position, made at
    block row i-1).  Committed tokens: x_1..x_n and the bonus p_n.
    With forced_n the count is imposed instead (cache bookkeeping tests).
    """
    D = len(drafts)
    if forced_n is None:
        n = 0
        while n < D and int(drafts[n]) == int(p[n]):
            n += 1
    else:
        if not 0 <= forced_n <= D:
            raise ValueError("forced_n out of range")
        n = int(forced_n)
    out = [int(t) for t in drafts[:n]] + [int(p[n])]
    return n, out


def commit(st: SeqState, n: int, out: Sequence[int], new_k, new_v) -> None:
    """Sec. 3 step 5: keep block rows 0..n (anchor, x_1..x_n) in the cache,
    drop the rest; the bonus token becomes the new anchor."""
    for li in range(len(st.cache_k)):
        st.cache_k[li] = np.concatenate([st.cache_k[li], new_k[li][: n + 1]], axis=0)
        st.cache_v[li] = np.concatenate([st.cache_v[li], new_v[li][: n + 1]], axis=0)
    st.anchor = int(out[-1])
    st.tokens.extend(int(t) for t in out)
    st.generated.extend(int(t) for t in out)


def step(model: OracleModel, st: SeqState, forced_n: Optional[int] = None):
    """One speculative step: draft, verify, accept, commit."""
    drafts, dlg = draft(model, st)
    p, vlg, k, v = verify(model, st, drafts)
    n, out = accept(drafts, p, forced_n)
    commit(st, n, out, k, v)
    return dict(drafts=drafts, draft_logits=dlg, p=p, verify_logits=vlg, n=n, out=out)


def generate(model: OracleModel, prompt: Sequence[int], budget: int,
             forced: Optional[Sequence[int]] = None):
    """Repeat speculative steps until `budget` tokens are generated (the first
    one comes from the prefill); the list is truncated to the budget."""
    st = prefill(model, prompt)
    rounds = []
    r = 0
    while len(st.generated) < budget:
        fn = None if forced is None else int(forced[r])
        info = step(model, st, fn)
        rounds.append(info["n"])
        r += 1
    return st.generated[:budget], rounds, st
