"""Decoder forward for the oracle: prefill that builds a KV cache, and one
decode step that extends it.

The paper rebuilds the prefix cache with the serving engine's ordinary
prefill (Sections 4.3 and 5) and resumes decoding at position n from the
assembled cache without re-running prefill (Section 4.3, "Final
synchronization and activation").  It names the model families (Llama-3,
Qwen3; Section 6.1) but not their arithmetic, so the forward below is the
standard pre-norm decoder of those families:

* RMSNorm x * (mean(x^2) + eps)^(-1/2) * g;
* fused Q|K|V projection, no biases;
* optional per-head RMSNorm of Q and K over the head dimension (Qwen3),
  applied before rotary embedding;
* rotary embedding on the two halves of each head, angle
  pos * theta^(-2i/d), absolute 0-based positions;
* causal grouped-query attention, query head h reads KV head h // (Hq/Hkv),
  scale 1/sqrt(d), exact softmax;
* SwiGLU MLP down(silu(gate) * up) with a fused gate|up projection;
* float residual stream; final RMSNorm and an untied output projection.

Arithmetic is float64; ``rnd`` rounds at the points where the model stores
bf16: normalised activations, the Q|K|V projection output, post-rotary Q and
K (the cache holds post-rotary K), the attention output and the SwiGLU
product.  Passing ``numerics.no_round`` gives the same forward unrounded.

Weights are float arrays: per layer ``attn_norm [H]``, ``w_qkv [(Hq+2Hkv)d,
H]`` (rows: Q heads, then K heads, then V heads), ``q_norm [d]``, ``k_norm
[d]``, ``w_o [H, Hq d]``, ``mlp_norm [H]``, ``w_gate_up [2F, H]`` (rows: gate,
then up), ``w_down [H, F]``; globally ``embed [V, H]``, ``final_norm [H]``,
``lm_head [V, H]``.  Matrices are [out, in].
"""
from __future__ import annotations

import math
from dataclasses import dataclass
from typing import Callable, Dict, List, Optional, Sequence

import numpy as np

from .numerics import bf16_round

Rounder = Callable[[np.ndarray], np.ndarray]


@dataclass(frozen=True)
class Shape:
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

    @staticmethod
    def of(cfg) -> "Shape":
        return Shape(cfg.n_layers, cfg.hidden, cfg.n_q_heads, cfg.n_kv_heads,
                     cfg.head_dim, cfg.ffn, cfg.vocab, bool(cfg.qk_norm),
                     float(cfg.rms_eps), float(cfg.rope_theta))


_DTYPE = np.float64


def f64(a) -> np.ndarray:
    """Cast to the working precision (float64 unless ``precision`` is active)."""
    return np.asarray(a, dtype=_DTYPE)


class precision:
    """Context manager that evaluates the forward in another floating type
    (float32 to measure how bf16 rounding decisions drift with depth when
    the arithmetic is float32 rather than float64).  The default is
    float64."""

    def __init__(self, dtype):
        self.dtype = dtype

    def __enter__(self):
        global _DTYPE
        self.saved, _DTYPE = _DTYPE, self.dtype
        return self

    def __exit__(self, *exc):
        global _DTYPE
        _DTYPE = self.saved
        return False


def rmsnorm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    """x * (mean(x^2) + eps)^(-1/2) * g over the last axis."""
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * g


def rope(x: np.ndarray, pos: np.ndarray, theta: float) -> np.ndarray:
    """Rotary embedding of ``x [T, heads, d]`` at positions ``pos [T]``:
    element i (i < d/2) pairs with element i + d/2 and the pair is rotated
    by pos * theta^(-2i/d)."""
    d = x.shape[-1]
    half = d // 2
    inv_freq = theta ** (-(2.0 * np.arange(half, dtype=np.float64)) / d)
    ang = np.asarray(pos, dtype=np.float64)[:, None] * inv_freq[None, :]
    c = f64(np.cos(ang))[:, None, :]
    s = f64(np.sin(ang))[:, None, :]
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def silu(x: np.ndarray) -> np.ndarray:
    return x / (1.0 + np.exp(-x))


def causal_attention(q: np.ndarray, q_pos: np.ndarray, k: np.ndarray,
                     v: np.ndarray) -> np.ndarray:
    """softmax(q k^T / sqrt(d) + causal mask) v, per query head.

    ``q [T, Hq, d]`` holds queries at positions ``q_pos``; ``k, v [S, Hkv,
    d]`` hold keys and values at positions 0..S-1.  A query at position i
    sees keys 0..i.  Query head h reads KV head h // (Hq / Hkv)."""
    T, Hq, d = q.shape
    S, Hkv, _ = k.shape
    G = Hq // Hkv
    key_pos = np.arange(S)
    visible = key_pos[None, :] <= np.asarray(q_pos)[:, None]
    out = np.empty((T, Hq, d), dtype=np.result_type(q, v))
    scale = 1.0 / math.sqrt(d)
    for h in range(Hq):
        kh = h // G
        s = (q[:, h, :] @ k[:, kh, :].T) * scale
        s = np.where(visible, s, -np.inf)
        s = s - s.max(axis=1, keepdims=True)
        p = np.exp(s)
        p = p / p.sum(axis=1, keepdims=True)
        out[:, h, :] = p @ v[:, kh, :]
    return out


def qkv_heads(h: np.ndarray, w: Dict, shp: Shape, pos: np.ndarray, rnd: Rounder):
    """Q|K|V projection, optional per-head Q/K RMSNorm, rotary embedding.
    Returns post-rotary ``q [T,Hq,d]``, ``k [T,Hkv,d]`` and ``v [T,Hkv,d]``,
    each rounded as stored."""
    T = h.shape[0]
    Hq, Hkv, d = shp.n_q_heads, shp.n_kv_heads, shp.head_dim
    qkv = rnd(h @ f64(w["w_qkv"]).T)
    q = qkv[:, :Hq * d].reshape(T, Hq, d)
    k = qkv[:, Hq * d:(Hq + Hkv) * d].reshape(T, Hkv, d)
    v = qkv[:, (Hq + Hkv) * d:].reshape(T, Hkv, d)
    if shp.qk_norm:
        q = rmsnorm(q, f64(w["q_norm"]), shp.rms_eps)
        k = rmsnorm(k, f64(w["k_norm"]), shp.rms_eps)
    q = rnd(rope(q, pos, shp.rope_theta))
    k = rnd(rope(k, pos, shp.rope_theta))
    return q, k, v


def layer(r: np.ndarray, pos: np.ndarray, k_prev: Optional[np.ndarray],
          v_prev: Optional[np.ndarray], w: Dict, shp: Shape, rnd: Rounder,
          kv_only: bool = False):
    """One decoder layer over tokens at consecutive positions ``pos`` whose
    residual rows are ``r [T, H]``.  ``k_prev, v_prev [n0, Hkv, d]`` are the
    cached K/V of positions 0..n0-1 (or None when n0 = 0).

    Returns ``(r_out, k, v)`` where k, v are this layer's K/V of the T
    tokens.  With ``kv_only`` the layer stops once K and V exist and r_out
    is None."""
    h = rnd(rmsnorm(r, f64(w["attn_norm"]), shp.rms_eps))
    q, k, v = qkv_heads(h, w, shp, pos, rnd)
    if kv_only:
        return None, k, v
    K = k if k_prev is None else np.concatenate([k_prev, k], axis=0)
    V = v if v_prev is None else np.concatenate([v_prev, v], axis=0)
    o = rnd(causal_attention(q, pos, K, V)).reshape(r.shape[0], -1)
    r = r + o @ f64(w["w_o"]).T
    h2 = rnd(rmsnorm(r, f64(w["mlp_norm"]), shp.rms_eps))
    gu = h2 @ f64(w["w_gate_up"]).T
    F = shp.ffn
    a = rnd(silu(gu[:, :F]) * gu[:, F:])
    r = r + a @ f64(w["w_down"]).T
    return r, k, v


def embed(ids: Sequence[int], glob: Dict) -> np.ndarray:
    return f64(np.asarray(glob["embed"])[np.asarray(ids, dtype=np.int64)])


def logits(r_rows: np.ndarray, glob: Dict, shp: Shape, rnd: Rounder = bf16_round) -> np.ndarray:
    h = rnd(rmsnorm(r_rows, f64(glob["final_norm"]), shp.rms_eps))
    return h @ f64(glob["lm_head"]).T


def prefill(ids: Sequence[int], glob: Dict, layers: List[Dict], shp: Shape,
            rnd: Rounder = bf16_round, full_last: bool = False,
            n_layers: Optional[int] = None):
    """Causal prefill of ``ids`` from position 0.

    Returns ``(K, V, r)``: per-layer lists of ``[T, Hkv, d]`` K and V arrays
    (post-rotary, rounded as stored) and the final residual ``r [T, H]``
    (None unless ``full_last``).  Without ``full_last`` the last layer stops
    once its K and V exist, which leaves every K and V unchanged.
    ``n_layers`` evaluates only the first layers (their K/V do not depend on
    the later ones)."""
    L = shp.n_layers if n_layers is None else n_layers
    pos = np.arange(len(ids))
    r = embed(ids, glob)
    K, V = [], []
    for l in range(L):
        kv_only = (l == L - 1) and not full_last
        r, k, v = layer(r, pos, None, None, layers[l], shp, rnd, kv_only=kv_only)
        K.append(k)
        V.append(v)
    return K, V, r


def prefill_chunk(ids: Sequence[int], start: int, K_cache: List[np.ndarray],
                  V_cache: List[np.ndarray], glob: Dict, layers: List[Dict], shp: Shape,
                  rnd: Rounder = bf16_round, n_layers: Optional[int] = None):
    """Chunked prefill (Section 4.5: the target interleaves prefix
    reconstruction with resident decoding by prefilling in chunks).

    The tokens ``ids`` sit at positions ``start .. start + T - 1``; each one
    attends causally to the cached positions ``0 .. start - 1``
    (``K_cache[l], V_cache[l]`` hold at least ``[start, Hkv, d]``) and to
    the chunk's tokens up to itself.  Returns per-layer ``[T, Hkv, d]`` K and
    V of the chunk (the last evaluated layer stops once they exist)."""
    L = shp.n_layers if n_layers is None else n_layers
    pos = start + np.arange(len(ids))
    r = embed(ids, glob)
    K, V = [], []
    for l in range(L):
        kp = K_cache[l][:start] if start > 0 else None
        vp = V_cache[l][:start] if start > 0 else None
        r, k, v = layer(r, pos, kp, vp, layers[l], shp, rnd, kv_only=(l == L - 1))
        K.append(k)
        V.append(v)
    return K, V


def decode(token: int, n: int, K_cache: List[np.ndarray], V_cache: List[np.ndarray],
           glob: Dict, layers: List[Dict], shp: Shape, rnd: Rounder = bf16_round):
    """One decode step: token ``token`` at position ``n`` attends to the
    cached positions 0..n-1 and to itself.

    ``K_cache[l], V_cache[l]`` hold ``[n, Hkv, d]``.  Returns ``(logits [V],
    k_new, v_new)`` with this token's per-layer K/V ``[1, Hkv, d]``."""
    pos = np.array([n])
    r = embed([token], glob)
    k_new, v_new = [], []
    for l in range(shp.n_layers):
        r, k, v = layer(r, pos, K_cache[l][:n], V_cache[l][:n], layers[l], shp, rnd)
        k_new.append(k)
        v_new.append(v)
    return logits(r, glob, shp, rnd)[0], k_new, v_new
