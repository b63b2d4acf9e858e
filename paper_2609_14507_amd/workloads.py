"""Seeded synthetic decode workloads shaped like the paper's evaluation models.

This module only draws inputs: it holds none of the method's arithmetic
(no softmax, no merge, no routing).  Both the HIP path and the oracle consume
the arrays produced here, so a parity test compares the two on the same bytes.

Shapes follow the models of the evaluation setup (Sec. 7.1): Qwen3-30B-A3B
(GQA, 32 query heads, 4 KV heads, head dim 128), Mixtral-8x7B (GQA, 32 query
heads, 8 KV heads) and DeepSeek-V2-Lite (MLA, 16 heads, a 512-wide compressed
latent plus a 64-wide decoupled RoPE key).  The paper's prompts come from
ShareGPT and its weights from the released checkpoints; neither is needed on
the hot path, which only sees their shapes, so standard-normal bf16 draws
stand in for both.

Recipe: a CPU ``torch.Generator`` seeded with the config's seed draws fp32
``randn`` values that are rounded to bf16 (round-to-nearest-even).  Draw order:
ragged lengths and split fractions (ragged config only), then the cache
(per sequence: K then V, or the latent rows), then per decode step the
queries followed by the new K/V rows.
"""
from __future__ import annotations

import dataclasses
import math
from typing import List, Optional

import numpy as np
import torch

GQA = 0
MLA = 1


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    kind: int                  # GQA or MLA
    batch: int
    n_q_heads: int
    n_kv_heads: int            # MLA: 1 (one shared latent per token)
    head_dim: int              # GQA key/value width; MLA: v_head_dim of the expansion
    latent_dim: int = 0        # MLA compressed latent width
    rope_dim: int = 0          # MLA decoupled RoPE key width
    nope_dim: int = 0          # MLA per-head non-RoPE query width before absorption
    context: int = 0           # fixed context length (0 when ragged)
    ragged_lo: int = 0         # ragged context range [lo, hi] (inclusive), uniform ints
    ragged_hi: int = 0
    cpu_share: float = 0.0     # r: CPU share of the sequence (fixed configs)
    share_lo: float = 0.0      # ragged configs: per-sequence share ~ U[lo, hi]
    share_hi: float = 0.0
    sweep: tuple = ()          # CPU shares swept over one cache without moving data
    steps: int = 1             # decode steps per measured run
    kv_std: float = 1.0
    seed: int = 0
    block_tokens: int = 64

    @property
    def group(self) -> int:
        return self.n_q_heads // self.n_kv_heads

    @property
    def row_elems(self) -> int:
        """bf16 elements of one cached token of one KV head (GQA: K or V row; MLA: latent+rope)."""
        if self.kind == MLA:
            return self.latent_dim + self.rope_dim
        return self.head_dim

    @property
    def token_bytes(self) -> int:
        """Algorithmic KV bytes of one cached token (all KV heads, K and V; MLA: one latent row)."""
        if self.kind == MLA:
            return 2 * (self.latent_dim + self.rope_dim)
        return 2 * 2 * self.n_kv_heads * self.head_dim

    @property
    def softmax_scale(self) -> float:
        if self.kind == MLA:
            return 1.0 / math.sqrt(self.nope_dim + self.rope_dim)
        return 1.0 / math.sqrt(self.head_dim)


C1 = Workload("tiny-gqa-b1-h8-kv2-L2048", GQA, batch=1, n_q_heads=8, n_kv_heads=2,
              head_dim=128, context=2048, cpu_share=0.5, seed=1)
C2 = Workload("qwen3-30b-a3b-b16-L32768", GQA, batch=16, n_q_heads=32, n_kv_heads=4,
              head_dim=128, context=32768, cpu_share=0.3, seed=2)
C3 = Workload("mixtral-8x7b-b4-L131072-sweep", GQA, batch=4, n_q_heads=32, n_kv_heads=8,
              head_dim=128, context=131072, cpu_share=0.0, sweep=(0.0, 0.25, 0.5, 0.75), seed=3)
C4 = Workload("deepseek-v2-lite-mla-b8-L65536", MLA, batch=8, n_q_heads=16, n_kv_heads=1,
              head_dim=128, latent_dim=512, rope_dim=64, nope_dim=128, context=65536,
              cpu_share=0.4, kv_std=0.5, seed=4)
C5 = Workload("qwen3-30b-a3b-b8-ragged-1M", GQA, batch=8, n_q_heads=32, n_kv_heads=4,
              head_dim=128, ragged_lo=98304, ragged_hi=163840, share_lo=0.1, share_hi=0.6,
              steps=64, seed=5)

CONFIGS = {"c1": C1, "c2": C2, "c3": C3, "c4": C4, "c5": C5}


def split_point(share: float, length: int) -> int:
    """Token index of the CPU/GPU boundary for a CPU share r: s = floor(r * L)."""
    return int(math.floor(share * length))


def bf16_bits(t: torch.Tensor) -> np.ndarray:
    """bf16 tensor -> numpy uint16 array of its raw bits (no arithmetic)."""
    assert t.dtype == torch.bfloat16
    return t.contiguous().view(torch.int16).numpy().view(np.uint16)


def draw_bf16(gen: torch.Generator, shape, std: float = 1.0) -> np.ndarray:
    """fp32 standard-normal draw scaled by std, rounded to bf16 (RNE); returned as raw bits."""
    x = torch.randn(*shape, generator=gen, dtype=torch.float32)
    if std != 1.0:
        x = x * std
    return bf16_bits(x.to(torch.bfloat16))


@dataclasses.dataclass
class Prefill:
    """The cache contents of a workload before decode, in token-major layout.

    GQA: ``k[b]`` and ``v[b]`` are uint16 bf16 bits of shape [L_b, Hkv, D].
    MLA: ``k[b]`` holds latent rows [L_b, latent+rope]; ``v`` is None.
    """
    lengths: List[int]
    splits: List[int]
    k: List[np.ndarray]
    v: Optional[List[np.ndarray]]
    gen: torch.Generator


def make_prefill(w: Workload, batch: Optional[int] = None, context: Optional[int] = None) -> Prefill:
    """Draw the prefilled cache.  ``batch``/``context`` shrink a workload for quick tests
    while keeping its head shapes and draw recipe."""
    gen = torch.Generator(device="cpu")
    gen.manual_seed(w.seed)
    B = w.batch if batch is None else batch
    if w.ragged_hi:
        lo, hi = w.ragged_lo, w.ragged_hi
        if context is not None:           # scale the ragged range down proportionally
            f = context / hi
            lo, hi = max(1, int(lo * f)), max(1, int(hi * f))
        lengths = torch.randint(lo, hi + 1, (B,), generator=gen).tolist()
        fr = (torch.rand(B, generator=gen, dtype=torch.float64) * (w.share_hi - w.share_lo) + w.share_lo).tolist()
        splits = [split_point(f_, L) for f_, L in zip(fr, lengths)]
    else:
        L = w.context if context is None else context
        lengths = [L] * B
        splits = [split_point(w.cpu_share, L)] * B
    ks, vs = [], []
    for b in range(B):
        if w.kind == MLA:
            ks.append(draw_bf16(gen, (lengths[b], w.row_elems), w.kv_std))
        else:
            ks.append(draw_bf16(gen, (lengths[b], w.n_kv_heads, w.head_dim), w.kv_std))
            vs.append(draw_bf16(gen, (lengths[b], w.n_kv_heads, w.head_dim), w.kv_std))
    return Prefill(lengths, splits, ks, vs if w.kind == GQA else None, gen)


@dataclasses.dataclass
class StepInputs:
    """One decode step's inputs (uint16 bf16 bits).

    GQA: q [B, Hq, D]; k_new, v_new [B, Hkv, D].
    MLA: q [B, H, latent+rope] is the absorbed query (q_lat | q_rope) handed to
    attend; q_nope [B, H, nope] and q_rope [B, H, rope] are the pre-absorption
    query parts; k_new [B, latent+rope]; v_new None.
    """
    q: np.ndarray
    k_new: np.ndarray
    v_new: Optional[np.ndarray]
    q_nope: Optional[np.ndarray] = None
    q_rope: Optional[np.ndarray] = None


def draw_step(w: Workload, gen: torch.Generator, batch: Optional[int] = None) -> StepInputs:
    B = w.batch if batch is None else batch
    if w.kind == MLA:
        q = draw_bf16(gen, (B, w.n_q_heads, w.row_elems))
        q_nope = draw_bf16(gen, (B, w.n_q_heads, w.nope_dim))
        q_rope = q[:, :, w.latent_dim:].copy()
        k_new = draw_bf16(gen, (B, w.row_elems), w.kv_std)
        return StepInputs(q, k_new, None, q_nope=q_nope, q_rope=q_rope)
    q = draw_bf16(gen, (B, w.n_q_heads, w.head_dim))
    k_new = draw_bf16(gen, (B, w.n_kv_heads, w.head_dim), w.kv_std)
    v_new = draw_bf16(gen, (B, w.n_kv_heads, w.head_dim), w.kv_std)
    return StepInputs(q, k_new, v_new)


def draw_mla_weights(w: Workload, gen: torch.Generator):
    """Synthetic per-head absorption weights for the MLA path (bf16 bits).

    w_uk [H, nope, latent]: maps a head's non-RoPE query into the latent space.
    w_uv [H, latent, v_head]: expands a head's latent output to its value width.
    Drawn N(0, 1/latent) so projected activations stay O(1).
    """
    std_uk = 1.0 / math.sqrt(w.nope_dim)
    std_uv = 1.0 / math.sqrt(w.latent_dim)
    w_uk = draw_bf16(gen, (w.n_q_heads, w.nope_dim, w.latent_dim), std_uk)
    w_uv = draw_bf16(gen, (w.n_q_heads, w.latent_dim, w.head_dim), std_uv)
    return w_uk, w_uv


def draw_cpu_partial(gen: torch.Generator, rows: int, width: int):
    """A synthetic stand-in for the CPU engine's partial (O, LSE) when only the
    merge kernel's cost is of interest: O ~ N(0, 0.1) fp32, LSE ~ 10 + N(0, 1) fp32."""
    o = torch.randn(rows, width, generator=gen, dtype=torch.float32) * 0.1
    lse = torch.randn(rows, generator=gen, dtype=torch.float32) + 10.0
    return o.numpy(), lse.numpy()
