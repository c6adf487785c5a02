"""Per-token KV-cache footprint (Section 2.1, Eq. 1; introduction footnote).

Pinned by the paper's own figures: 262,144 bytes per token for 64 layers,
8 KV heads, head dimension 128 and 2-byte elements; about 1 GiB at 4000
tokens; about 28 s to send that at 300 Mbps; and the Full-Copy rows of
Table 1, which are transfer-bound.
"""


def s_kv(n_layers: int, n_kv_heads: int, head_dim: int, elem_bytes: int) -> int:
    """Eq. 1: s_KV = 2 * L * H_KV * d_h * b (K and V of every layer)."""
    return 2 * n_layers * n_kv_heads * head_dim * elem_bytes


def cache_bytes(n_tokens: int, n_layers: int, n_kv_heads: int, head_dim: int,
                elem_bytes: int) -> int:
    """Eq. 1: S_KV(N) = N * s_KV."""
    return n_tokens * s_kv(n_layers, n_kv_heads, head_dim, elem_bytes)


def transfer_seconds(n_bytes: int, goodput_bits_per_s: float) -> float:
    """Payload time over a link of the given goodput (the introduction's
    28-second example; the Full-Copy rows of Table 1)."""
    return n_bytes * 8.0 / goodput_bits_per_s


def copy_traffic_bytes(n_tokens: int, n_layers: int, n_kv_heads: int,
                       head_dim: int, elem_bytes: int) -> int:
    """Device-memory bytes one pack (or one assemble) of ``n_tokens`` moves:
    the payload read once and written once."""
    return 2 * cache_bytes(n_tokens, n_layers, n_kv_heads, head_dim, elem_bytes)
