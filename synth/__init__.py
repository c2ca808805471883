"""Seeded synthetic inputs for the PEFT-BD speculative step.

This module is shared by the CPU oracle and the GPU path and holds none of the
method's arithmetic: it only describes model shapes and draws random numbers.

* Model shapes: the paper evaluates Qwen3-0.6B (Sec. 4.1) with a LoRA-like
  adapter of rank 16, alpha 32 on every linear projection of every block
  (App. A.2); block size D = 16 (Sec. 3).  The paper prints no architecture, so
  the Qwen3-0.6B shape (28 layers, hidden 1024, 16/8 heads of dim 128, SwiGLU
  3072, vocab 151936, tied embeddings, per-head QK RMSNorm) is taken as the
  public model card states it.  A tiny fp32 decoder of the same structure
  serves for exact parity work.
* Weights: linear, embedding and LoRA weights ~ N(0, 0.02); norm gains
  1 + N(0, 0.02) so the gain multiply is observable; drawn in one fixed
  canonical order from numpy ``Generator(PCG64(seed))`` and rounded to bf16
  (round-to-nearest-even) for bf16 models, so both sides read the same values.
* Prompts: token ids uniform on [0, V-1) (the mask id V-1 never appears);
  ragged prefix lengths uniform on an integer range.
* Forced acceptance: committed tokens per round n+1 ~ Geometric(1/3) on
  {1, 2, ...} truncated at D+1 (mean 3, close to the 2.881 committed tokens
  per round of the paper's Tab. uncertainty).
"""
from __future__ import annotations

import dataclasses
from dataclasses import dataclass, field
from typing import List, Optional, Tuple

import numpy as np

# Order of the seven adapted projections of one transformer block (App. A.2:
# LoRA on all attention and MLP projection modules).
LORA_TARGETS = ("q", "k", "v", "o", "gate", "up", "down")


@dataclass(frozen=True)
class ModelConfig:
    name: str
    n_layers: int
    hidden: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    ffn: int
    vocab: int
    lora_rank: int
    lora_alpha: float
    block: int = 16              # D, masked positions per draft (Sec. 3)
    rms_eps: float = 1e-6
    rope_theta: float = 1e6
    qk_norm: bool = True
    dtype: str = "bf16"          # "f32" or "bf16": weights, KV cache, GEMM inputs

    @property
    def mask_id(self) -> int:
        # The diffusion mask token is the last vocabulary row (a padded row of
        # the embedding table, trained in the paper, random here).
        return self.vocab - 1

    @property
    def width(self) -> int:
        # Pass width W = D + 1: the anchor plus D masks (draft) or D drafts
        # (verify); "token width 17" in Tab. profile.
        return self.block + 1

    @property
    def lora_scale(self) -> float:
        return self.lora_alpha / self.lora_rank

    def with_(self, **kw) -> "ModelConfig":
        return dataclasses.replace(self, **kw)

    def linear_shapes(self):
        """(name, out_features, in_features) for the seven block projections."""
        H, d = self.hidden, self.head_dim
        return (
            ("q", self.n_q_heads * d, H),
            ("k", self.n_kv_heads * d, H),
            ("v", self.n_kv_heads * d, H),
            ("o", H, self.n_q_heads * d),
            ("gate", self.ffn, H),
            ("up", self.ffn, H),
            ("down", H, self.ffn),
        )


TINY = ModelConfig(
    name="tiny-fp32", n_layers=2, hidden=256, n_q_heads=4, n_kv_heads=2,
    head_dim=64, ffn=768, vocab=4096, lora_rank=8, lora_alpha=16.0,
    dtype="f32",
)

QWEN3_0_6B = ModelConfig(
    name="qwen3-0.6b", n_layers=28, hidden=1024, n_q_heads=16, n_kv_heads=8,
    head_dim=128, ffn=3072, vocab=151936, lora_rank=16, lora_alpha=32.0,
    dtype="bf16",
)


@dataclass(frozen=True)
class Workload:
    """One benchmark/parity workload: a model plus its batch of sequences."""
    index: int
    name: str
    cfg: ModelConfig
    batch: int
    prefix: Tuple[int, int]      # prefix length range [lo, hi] (lo == hi: fixed)
    gen_tokens: int = 0          # >0: generation loop budget (tokens)
    description: str = ""

    def seed(self, stream: int) -> int:
        # stream: 0 weights, 1 prompt tokens, 2 ragged lengths, 3 forced n
        return 1000 * self.index + stream


WORKLOADS: List[Workload] = [
    Workload(0, "tiny-fp32-b1-p128", TINY, 1, (128, 128),
             description="tiny fp32 decoder, prefix 128, one D=16 draft+verify step"),
    Workload(1, "qwen3-0.6b-b1-p512", QWEN3_0_6B, 1, (512, 512),
             description="Qwen3-0.6B shape bf16, r=16, prefix 512, one D=16 step"),
    Workload(2, "qwen3-0.6b-b1-p4096-gen256", QWEN3_0_6B, 1, (4096, 4096), 256,
             description="prefix 4096, loop of 256 generated tokens"),
    Workload(3, "qwen3-0.6b-b8-ragged", QWEN3_0_6B.with_(lora_rank=32, lora_alpha=64.0),
             8, (256, 2048),
             description="batch 8, prefixes uniform in [256, 2048], r=32"),
    Workload(4, "qwen3-0.6b-b32-p8192-d32", QWEN3_0_6B.with_(lora_rank=64, lora_alpha=128.0,
                                                            block=32),
             32, (8192, 8192),
             description="batch 32, prefix 8192, D=32, r=64"),
]


def round_bf16(x: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bf16 (ties to even); returns float32."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    bits = x.view(np.uint32)
    lsb = (bits >> 16) & 1
    rounded = ((bits + np.uint32(0x7FFF) + lsb) & np.uint32(0xFFFF0000)).astype(np.uint32)
    return rounded.view(np.float32)


@dataclass
class LayerWeights:
    attn_norm: np.ndarray
    q: np.ndarray
    k: np.ndarray
    v: np.ndarray
    o: np.ndarray
    q_norm: np.ndarray
    k_norm: np.ndarray
    mlp_norm: np.ndarray
    gate: np.ndarray
    up: np.ndarray
    down: np.ndarray
    lora: dict = field(default_factory=dict)   # name -> (A [r][in], B [out][r])


@dataclass
class Weights:
    cfg: ModelConfig
    embed: np.ndarray            # [V][H], tied with the LM head
    layers: List[LayerWeights]
    final_norm: np.ndarray       # [H]


def make_weights(cfg: ModelConfig, seed: int, zero_lora_b: bool = False) -> Weights:
    """Draw every weight in the fixed canonical order (float32 arrays).

    Order: E; per layer attn_norm, q, k, v, o, q_norm, k_norm, mlp_norm, gate,
    up, down, then (A, B) for q, k, v, o, gate, up, down; final_norm.
    ``zero_lora_b`` still draws B (so the stream is unchanged) but zeroes it.
    """
    rng = np.random.Generator(np.random.PCG64(seed))
    H, d, F = cfg.hidden, cfg.head_dim, cfg.ffn
    r = cfg.lora_rank
    rnd = (lambda a: round_bf16(a)) if cfg.dtype == "bf16" else (lambda a: a)

    def lin(o, i):
        return rnd((rng.standard_normal((o, i), dtype=np.float32) * np.float32(0.02)))

    def gain(n):
        return rnd(np.float32(1.0) + rng.standard_normal(n, dtype=np.float32) * np.float32(0.02))

    embed = lin(cfg.vocab, H)
    layers = []
    shapes = {n: (o, i) for n, o, i in cfg.linear_shapes()}
    for _ in range(cfg.n_layers):
        attn_norm = gain(H)
        q = lin(*shapes["q"]); k = lin(*shapes["k"]); v = lin(*shapes["v"])
        o = lin(*shapes["o"])
        q_norm = gain(d); k_norm = gain(d)
        mlp_norm = gain(H)
        gate = lin(*shapes["gate"]); up = lin(*shapes["up"]); down = lin(*shapes["down"])
        lora = {}
        for name in LORA_TARGETS:
            out_f, in_f = shapes[name]
            A = lin(r, in_f)
            B = lin(out_f, r)
            if zero_lora_b:
                B = np.zeros_like(B)
            lora[name] = (A, B)
        layers.append(LayerWeights(attn_norm, q, k, v, o, q_norm, k_norm, mlp_norm,
                                   gate, up, down, lora))
    final_norm = gain(H)
    return Weights(cfg, embed, layers, final_norm)


def make_prompts(cfg: ModelConfig, lengths: List[int], seed: int) -> List[np.ndarray]:
    """Prompt token ids uniform on [0, V-1) (never the mask id)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    return [rng.integers(0, cfg.vocab - 1, size=n, dtype=np.int64).astype(np.int32)
            for n in lengths]


def make_lengths(batch: int, lo: int, hi: int, seed: int) -> List[int]:
    if lo == hi:
        return [lo] * batch
    rng = np.random.Generator(np.random.PCG64(seed))
    return [int(x) for x in rng.integers(lo, hi + 1, size=batch)]


def make_forced_accepts(n_rounds: int, batch: int, block: int, seed: int,
                        mean_commit: float = 3.0) -> np.ndarray:
    """Forced accepted-draft counts n in [0, D]: n+1 ~ Geometric(1/mean) truncated at D+1."""
    rng = np.random.Generator(np.random.PCG64(seed))
    commits = rng.geometric(1.0 / mean_commit, size=(n_rounds, batch))
    return (np.minimum(commits, block + 1) - 1).astype(np.int32)


def workload_inputs(w: Workload, batch: Optional[int] = None):
    """(lengths, prompts) for a workload; ``batch`` may take a leading subset."""
    lengths = make_lengths(w.batch, w.prefix[0], w.prefix[1], w.seed(2))
    prompts = make_prompts(w.cfg, lengths, w.seed(1))
    if batch is not None:
        lengths, prompts = lengths[:batch], prompts[:batch]
    return lengths, prompts
