"""Oracle pins: the per-token KV footprint (Eq. 1) against the paper's own
printed figures (introduction footnote, the 1 GiB / 28 s example, Table 1's
transfer-bound Full-Copy rows)."""
import json
import os

import pytest

from oracle import footprint
from workloads import configs

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "kv_footprint.json")))


def test_s_kv_matches_footnote():
    m = GOLD["qwen3_32b"]
    s = footprint.s_kv(m["n_layers"], m["n_kv_heads"], m["head_dim"], m["elem_bytes"])
    assert s == GOLD["s_kv_bytes_per_token"]
    assert s == GOLD["approx_kib_per_token"] * 1024


def test_cache_size_and_transfer_time_example():
    m = GOLD["qwen3_32b"]
    b = footprint.cache_bytes(GOLD["tokens_example"], m["n_layers"], m["n_kv_heads"],
                              m["head_dim"], m["elem_bytes"])
    assert b == 4000 * 262144
    assert abs(b / 2**30 - GOLD["approx_gib_at_example"]) < 0.05
    t = footprint.transfer_seconds(b, GOLD["goodput_mbps"] * 1e6)
    assert abs(t - GOLD["approx_transfer_s_at_example"]) < 0.5


@pytest.mark.parametrize("tokens", ["1024", "2048", "4096"])
def test_full_copy_rows_are_transfer_bound(tokens):
    """Table 1's Full-Copy recovery is the cache payload over 300 Mbps."""
    m = GOLD["qwen3_32b"]
    b = footprint.cache_bytes(int(tokens), m["n_layers"], m["n_kv_heads"],
                              m["head_dim"], m["elem_bytes"])
    t_ms = footprint.transfer_seconds(b, GOLD["goodput_mbps"] * 1e6) * 1e3
    measured = GOLD["table1_full_copy_ms"][tokens]
    assert abs(t_ms - measured) / measured < 0.025


def test_preset_footprints():
    assert configs.LARGE.s_kv == 262144
    assert configs.MID.s_kv == 147456
    assert configs.TINY.s_kv == 1024


@pytest.mark.parametrize("n,start", [(1000, 3000), (37, 5)])
def test_copy_traffic_is_the_packed_payload_read_and_written(n, start):
    """copy_traffic_bytes against what a pack actually moves: the oracle's
    brute-force pack of n tokens out of a paged pool yields a chunk whose
    bytes numpy counts from its shape; each of them is read once from the
    pool and written once, so the traffic is twice the chunk.  At the large
    shape and 1000 tokens that is the 524.3 MB of the copy metric."""
    import numpy as np
    from oracle import paged
    L, hkv, d = (64, 8, 128) if n == 1000 else (3, 2, 16)
    pages = (start + n + 15) // 16
    pool = np.zeros((L, 2, pages, 16, hkv, d), np.uint16)
    bt = np.arange(pages)[::-1].copy()
    chunk = paged.pack(pool, bt, start, n)
    assert footprint.copy_traffic_bytes(n, L, hkv, d, 2) == 2 * chunk.nbytes
    if n == 1000:
        assert 2 * chunk.nbytes == 524288000


def test_prefill_flop_count():
    # 64.56 GFLOP/token at the large shape over a 3000-token prefix
    f = configs.LARGE.prefill_flops(3000)
    assert abs(f / 3000 / 1e9 - 64.56) < 0.05
    f2 = configs.MID.prefill_flops(1536)
    assert abs(f2 / 1536 / 1e9 - 13.96) < 0.05
