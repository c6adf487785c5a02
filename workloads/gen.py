"""Deterministic synthetic inputs.

Every tensor is drawn from its own stream, keyed by (seed, workload tag,
layer, tensor id), so one layer can be regenerated without the others.
Matrices and embeddings are N(0, 0.02) rounded to bf16 (round to nearest
even, torch's conversion); RMSNorm gains are 1 unless ``gain_sigma`` is
given, in which case they are 1 + N(0, gain_sigma).  Token ids are uniform
over the vocabulary; block tables are seeded permutations of free pages.

Streams use torch generators on the requested device, so a tensor drawn on
the GPU differs from the same key drawn on the CPU.  Consumers that need the
same bytes on both sides (the oracle and the HIP path) draw once and copy.
"""
from __future__ import annotations

from typing import Dict, List, Optional

import numpy as np
import torch

from .configs import ModelConfig

# Tensor ids inside a layer.
LAYER_TENSORS = ("attn_norm", "w_qkv", "q_norm", "k_norm", "w_o", "mlp_norm",
                 "w_gate_up", "w_down")
GLOBAL_TENSORS = ("embed", "final_norm", "lm_head")
SIGMA = 0.02


def stream_seed(*keys: int) -> int:
    ss = np.random.SeedSequence([int(k) & 0xFFFFFFFF for k in keys])
    return int(ss.generate_state(1, dtype=np.uint64)[0] & ((1 << 63) - 1))


def torch_gen(device, *keys: int) -> torch.Generator:
    dev = torch.device(device)
    g = torch.Generator(device=dev)
    g.manual_seed(stream_seed(*keys))
    return g


def normal_bf16(shape, sigma: float, device, *keys: int, mean: float = 0.0) -> torch.Tensor:
    g = torch_gen(device, *keys)
    x = torch.randn(*shape, generator=g, device=device, dtype=torch.float32)
    if sigma != 1.0:
        x.mul_(sigma)
    if mean != 0.0:
        x.add_(mean)
    return x.to(torch.bfloat16)


def layer_shapes(cfg: ModelConfig) -> Dict[str, tuple]:
    H, d, F = cfg.hidden, cfg.head_dim, cfg.ffn
    return {
        "attn_norm": (H,),
        "w_qkv": (cfg.qkv_out, H),
        "q_norm": (d,),
        "k_norm": (d,),
        "w_o": (H, cfg.q_dim),
        "mlp_norm": (H,),
        "w_gate_up": (2 * F, H),
        "w_down": (H, F),
    }


def global_shapes(cfg: ModelConfig) -> Dict[str, tuple]:
    return {"embed": (cfg.vocab, cfg.hidden), "final_norm": (cfg.hidden,),
            "lm_head": (cfg.vocab, cfg.hidden)}


_GAINS = ("attn_norm", "q_norm", "k_norm", "mlp_norm", "final_norm")


def _draw(name: str, shape, device, seed: int, tag: int, layer: int, tid: int,
          gain_sigma: Optional[float]) -> torch.Tensor:
    if name in _GAINS:
        if gain_sigma is None:
            return torch.ones(shape, dtype=torch.bfloat16, device=device)
        return normal_bf16(shape, gain_sigma, device, seed, tag, layer, tid, mean=1.0)
    return normal_bf16(shape, SIGMA, device, seed, tag, layer, tid)


def layer_weights(cfg: ModelConfig, layer: int, seed: int = 0, tag: int = 0,
                  device="cpu", gain_sigma: Optional[float] = None) -> Dict[str, torch.Tensor]:
    shapes = layer_shapes(cfg)
    return {name: _draw(name, shapes[name], device, seed, tag, layer, tid, gain_sigma)
            for tid, name in enumerate(LAYER_TENSORS)}


def global_weights(cfg: ModelConfig, seed: int = 0, tag: int = 0, device="cpu",
                   gain_sigma: Optional[float] = None) -> Dict[str, torch.Tensor]:
    shapes = global_shapes(cfg)
    return {name: _draw(name, shapes[name], device, seed, tag, 0xFFFF, tid, gain_sigma)
            for tid, name in enumerate(GLOBAL_TENSORS)}


def model_weights(cfg: ModelConfig, seed: int = 0, tag: int = 0, device="cpu",
                  gain_sigma: Optional[float] = None):
    """All weights: ``(globals, [layer dicts])`` as bf16 tensors on ``device``."""
    glob = global_weights(cfg, seed, tag, device, gain_sigma)
    layers = [layer_weights(cfg, l, seed, tag, device, gain_sigma)
              for l in range(cfg.n_layers)]
    return glob, layers


def token_ids(n: int, vocab: int, seed: int = 0, tag: int = 0, stream: int = 0) -> torch.Tensor:
    """``n`` ids uniform over ``[0, vocab)`` (int32, CPU)."""
    g = torch_gen("cpu", seed, tag, 0xA11D, stream)
    return torch.randint(0, vocab, (n,), generator=g, dtype=torch.int64).to(torch.int32)


def permutation(n: int, seed: int, *keys: int) -> np.ndarray:
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence(
        [seed, 0xB10C] + [int(k) for k in keys])))
    return rng.permutation(n).astype(np.int32)


def block_table(pages_needed: int, pool_pages: int, max_pages: int, seed: int,
                *keys: int, free_pages: Optional[np.ndarray] = None) -> np.ndarray:
    """A block table of ``max_pages`` entries: the first ``pages_needed`` are
    distinct pages of the pool (drawn in seeded order from ``free_pages`` or
    the whole pool), the rest are -1."""
    if free_pages is None:
        free_pages = np.arange(pool_pages, dtype=np.int32)
    assert pages_needed <= len(free_pages) and pages_needed <= max_pages
    order = permutation(len(free_pages), seed, *keys)
    bt = np.full(max_pages, -1, dtype=np.int32)
    bt[:pages_needed] = np.asarray(free_pages, dtype=np.int32)[order[:pages_needed]]
    return bt


def disjoint_block_tables(pages: List[int], pool_pages: int, max_pages: int,
                          seed: int, *keys: int) -> np.ndarray:
    """Tables for several sequences over one shared pool: every sequence gets
    its own pages, all drawn from one seeded permutation of the pool."""
    assert sum(pages) <= pool_pages
    order = permutation(pool_pages, seed, *keys)
    out = np.full((len(pages), max_pages), -1, dtype=np.int32)
    off = 0
    for i, n in enumerate(pages):
        out[i, :n] = order[off:off + n]
        off += n
    return out


def kv_pool_normal(n_layers: int, num_pages: int, page: int, n_kv_heads: int,
                   head_dim: int, seed: int, device="cpu", tag: int = 4) -> torch.Tensor:
    """A pool ``bf16 [L][2][P][page][Hkv][d]`` filled with N(0, 1)."""
    shape = (n_layers, 2, num_pages, page, n_kv_heads, head_dim)
    return normal_bf16(shape, 1.0, device, seed, tag, 0xF00D, 0)


SENTINEL_BITS = 0x7FA5  # a quiet-NaN bf16 pattern that no N(0,1) draw produces
