"""Paged KV cache, suffix-block extraction and target-side assembly.

The prototype keeps each request's KV cache in 16-token PagedAttention
blocks addressed through a block table (Section 5).  During preparation the
source extracts the per-layer K/V tensors of completed suffix blocks and
streams them with their logical token positions (Section 4.3,
"Initialization and parallel preparation"; Section 5); at handover the target
allocates a new block table and copies the prefix and the buffered suffix
into it (Section 5, "Final synchronization and activation"), after checking
that the cache covers every position of [0, n) with no gap or conflict and
that no block of a cancelled attempt (an older migration epoch) enters the
request (Section 4.3, "State consistency"; Section 4.4).

Layouts (fixed by the library boundary and mirrored here):

* pool  ``[L, 2, P, page, Hkv, d]``: layer, K|V, page, slot, head, dim;
* block table ``[max_pages]``: logical page -> physical page (-1 unused);
* chunk ``[L, 2, count, Hkv, d]``: the K/V of ``count`` consecutive
  positions starting at ``start``, contiguous per layer.

Arrays may hold any element type; copies are bit-for-bit.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import List, Sequence

import numpy as np


def logical_view(pool: np.ndarray, bt: np.ndarray, n: int) -> np.ndarray:
    """``out[l, kv, t] = pool[l, kv, bt[t // page], t % page]`` for t < n."""
    page = pool.shape[3]
    t = np.arange(n)
    return pool[:, :, np.asarray(bt)[t // page], t % page]


def write_positions(pool: np.ndarray, bt: np.ndarray, start: int, kv: np.ndarray) -> None:
    """Store ``kv [L, 2, T, Hkv, d]`` at positions start..start+T-1."""
    page = pool.shape[3]
    t = start + np.arange(kv.shape[2])
    pool[:, :, np.asarray(bt)[t // page], t % page] = kv


def write_cache(pool: np.ndarray, bt: np.ndarray, K: List[np.ndarray],
                V: List[np.ndarray], start: int = 0) -> None:
    """Store per-layer ``K[l], V[l] [T, Hkv, d]`` (a prefill's output)."""
    kv = np.stack([np.stack([K[l], V[l]]) for l in range(len(K))])
    write_positions(pool, bt, start, kv.astype(pool.dtype))


def pack(pool: np.ndarray, bt: np.ndarray, start: int, count: int) -> np.ndarray:
    """Suffix-block extraction: the chunk of positions [start, start+count)."""
    page = pool.shape[3]
    t = start + np.arange(count)
    return pool[:, :, np.asarray(bt)[t // page], t % page].copy()


@dataclass
class ChunkHeader:
    request_id: int
    epoch: int
    start_pos: int
    num_tokens: int
    n_layers: int
    n_kv_heads: int
    head_dim: int
    elem_bytes: int


class Rejected(Exception):
    """Assembly refused before anything was written; ``code`` names why."""

    def __init__(self, code: str, msg: str):
        super().__init__(f"{code}: {msg}")
        self.code = code


def check_chunks(pool: np.ndarray, table_capacity: int, hdrs: Sequence[ChunkHeader],
                 expected_request_id: int, expected_epoch: int) -> None:
    """The host-side checks of assembly, in this order: shape, request id,
    epoch, range inside the table, no two chunks claiming one position."""
    L, _, _, _, Hkv, d = pool.shape
    eb = pool.dtype.itemsize
    for h in hdrs:
        if (h.n_layers, h.n_kv_heads, h.head_dim, h.elem_bytes) != (L, Hkv, d, eb):
            raise Rejected("INVALID_ARG", "chunk shape differs from the pool")
    for h in hdrs:
        if h.request_id != expected_request_id:
            raise Rejected("WRONG_REQUEST", "chunk belongs to another request")
    for h in hdrs:
        if h.epoch != expected_epoch:
            raise Rejected("STALE_EPOCH", "chunk comes from another migration epoch")
    for h in hdrs:
        if h.start_pos < 0 or h.num_tokens < 0 or h.start_pos + h.num_tokens > table_capacity:
            raise Rejected("OUT_OF_RANGE", "chunk range outside the block table")
    spans = sorted((h.start_pos, h.start_pos + h.num_tokens) for h in hdrs if h.num_tokens > 0)
    for (a0, a1), (b0, b1) in zip(spans, spans[1:]):
        if b0 < a1:
            raise Rejected("COVERAGE", "two chunks claim the same position")


def assemble(pool: np.ndarray, bt: np.ndarray, hdrs: Sequence[ChunkHeader],
             chunks: Sequence[np.ndarray], expected_request_id: int,
             expected_epoch: int) -> bool:
    """Scatter each chunk into the pool through the target block table.

    Raises ``Rejected`` (pool untouched) when a host-side check fails.  A
    position whose table entry names no page of the pool is skipped; the
    return value is False when that happened, True otherwise."""
    bt = np.asarray(bt)
    page = pool.shape[3]
    P = pool.shape[2]
    check_chunks(pool, len(bt) * page, hdrs, expected_request_id, expected_epoch)
    clean = True
    for h, c in zip(hdrs, chunks):
        for i in range(h.num_tokens):
            t = h.start_pos + i
            pg = int(bt[t // page])
            if pg < 0 or pg >= P:
                clean = False
                continue
            pool[:, :, pg, t % page] = c[:, :, i]
    return clean


def check_coverage(prefix_len: int, starts: Sequence[int], lens: Sequence[int], n: int) -> bool:
    """True iff [0, prefix_len) and the ranges [s, s+len) together cover
    [0, n) exactly once: no gap, no position claimed twice, nothing past n."""
    if prefix_len < 0 or prefix_len > n:
        return False
    spans = sorted((int(s), int(s) + int(c)) for s, c in zip(starts, lens))
    at = prefix_len
    for s, e in spans:
        if e < s or s < 0:
            return False
        if s == e:
            continue
        if s != at:
            return False
        at = e
    return at == n
