"""Model-shape presets and request workloads.

Shapes follow the Qwen3-like decoders the paper evaluates (Section 6.1:
Llama-3-8B, Qwen3-14B, Qwen3-32B) and its per-token KV footprint (Eq. 1 and
the introduction's footnote: 64 layers, 8 KV heads, head dimension 128, two
bytes per element).  Page size 16 follows the prototype's PagedAttention
block size (Section 5).  Weights are random-init, not trained checkpoints.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, List, Optional

import numpy as np

PAGE = 16


@dataclasses.dataclass(frozen=True)
class ModelConfig:
    name: str
    n_layers: int
    hidden: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    ffn: int
    vocab: int
    qk_norm: bool
    rms_eps: float = 1e-6
    rope_theta: float = 1e6
    page_size: int = PAGE
    elem_bytes: int = 2

    @property
    def group(self) -> int:
        return self.n_q_heads // self.n_kv_heads

    @property
    def qkv_out(self) -> int:
        return (self.n_q_heads + 2 * self.n_kv_heads) * self.head_dim

    @property
    def q_dim(self) -> int:
        return self.n_q_heads * self.head_dim

    @property
    def kv_dim(self) -> int:
        return self.n_kv_heads * self.head_dim

    @property
    def s_kv(self) -> int:
        """Eq. 1: bytes of K and V per token over all layers."""
        return 2 * self.n_layers * self.n_kv_heads * self.head_dim * self.elem_bytes

    @property
    def page_bytes(self) -> int:
        """Bytes of one page of one layer's K (or V)."""
        return self.page_size * self.n_kv_heads * self.head_dim * self.elem_bytes

    def weight_bytes(self) -> int:
        H, F, V = self.hidden, self.ffn, self.vocab
        per_layer = (2 * H + self.qkv_out * H + 2 * self.head_dim + H * self.q_dim
                     + 2 * F * H + H * F)
        return 2 * (self.n_layers * per_layer + 2 * V * H + H)

    def prefill_flops(self, p: int) -> float:
        """Algorithmic FLOPs of a prefix prefill over ``p`` tokens of one
        sequence: every layer but the last runs the full block with
        causal-only attention; the last layer runs only the K/V projection."""
        H, F, d = self.hidden, self.ffn, self.head_dim
        Hq, Hkv = self.n_q_heads, self.n_kv_heads
        full = (2 * p * H * (Hq + 2 * Hkv) * d + 2 * p * Hq * d * H
                + 4 * p * H * F + 2 * p * F * H + 2 * Hq * d * p * (p + 1))
        last = 2 * p * H * 2 * Hkv * d
        return float((self.n_layers - 1) * full + last)

    def with_layers(self, n_layers: int) -> "ModelConfig":
        return dataclasses.replace(self, n_layers=n_layers,
                                   name=f"{self.name}-L{n_layers}")

    def replace(self, **kw) -> "ModelConfig":
        return dataclasses.replace(self, **kw)


# Named model shapes.
TINY = ModelConfig("tiny", n_layers=2, hidden=256, n_q_heads=4, n_kv_heads=2,
                   head_dim=64, ffn=688, vocab=1024, qk_norm=False)
MID = ModelConfig("mid", n_layers=36, hidden=4096, n_q_heads=32, n_kv_heads=8,
                  head_dim=128, ffn=12288, vocab=151936, qk_norm=True)
LARGE = ModelConfig("large", n_layers=64, hidden=5120, n_q_heads=64, n_kv_heads=8,
                    head_dim=128, ffn=25600, vocab=151936, qk_norm=True)

PRESETS: Dict[str, ModelConfig] = {"tiny": TINY, "mid": MID, "large": LARGE}


def preset(name: str) -> ModelConfig:
    return PRESETS[name]


@dataclasses.dataclass
class Workload:
    """One reconstruction workload: the context of each request, its split,
    and the page pools on either side."""
    name: str
    model: ModelConfig
    ctx: List[int]          # n_i: tokens held by the source at handover
    prefix: List[int]       # p_i: tokens rebuilt by target-side prefill
    chunk_tokens: Optional[int] = None   # suffix chunk size (None: one chunk)

    @property
    def num_seqs(self) -> int:
        return len(self.ctx)

    def suffix(self, i: int) -> int:
        return self.ctx[i] - self.prefix[i]

    def pages_for(self, tokens: int) -> int:
        return (tokens + self.model.page_size - 1) // self.model.page_size


def workload(name: str) -> Workload:
    """The five reconstruction workloads.

    tiny:    2-layer decoder, one 128-token request split at 96.
    mid:     36-layer decoder, one 2048-token request split at 1536.
    large:   64-layer decoder, one 4000-token request split at 3000
             (3000 is not a multiple of 16: page 187 is shared by the
             prefix and the suffix).
    large-aligned: as ``large`` split at 2992, the last complete page.
    concurrent: mid decoder, 8 requests, ctx log-uniform in [1000, 8000],
             prefix fraction uniform in [0.5, 0.9], split rounded down to a
             page boundary, suffix streamed in 32-token chunks.
    """
    if name == "tiny":
        return Workload(name, TINY, [128], [96])
    if name == "mid":
        return Workload(name, MID, [2048], [1536])
    if name == "large":
        return Workload(name, LARGE, [4000], [3000])
    if name == "large-aligned":
        return Workload(name, LARGE, [4000], [2992])
    if name == "concurrent":
        ctx, pre = concurrent_lengths(seed=0, n=8)
        return Workload(name, MID, ctx, pre, chunk_tokens=32)
    raise KeyError(name)


def concurrent_lengths(seed: int, n: int = 8, lo: int = 1000, hi: int = 8000,
                       fmin: float = 0.5, fmax: float = 0.9):
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 5, 0xC0])))
    ctx = np.floor(np.exp(rng.uniform(math.log(lo), math.log(hi), size=n))).astype(int)
    f = rng.uniform(fmin, fmax, size=n)
    pre = (16 * np.floor(f * ctx / 16)).astype(int)
    pre = np.maximum(pre, 16)
    return [int(c) for c in ctx], [int(p) for p in pre]


# Stress workload for the copy kernels: 64-layer / 8-head / d=128 KV pages.
STRESS_KV = LARGE
STRESS_SOURCE_TOKENS = 8192
STRESS_SUFFIXES = (64, 256, 1024, 4096)
STRESS_TARGET_PAGES = 1024
STRESS_CHUNK = 32
