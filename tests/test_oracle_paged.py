"""Oracle pins for the paged cache, suffix extraction, assembly and the
consistency checks (Sections 4.3, 4.4 and 5): brute-force element loops on
tiny pools, round trips, untouched sentinel pages, the all-or-nothing
rejection rules, and assembly reproducing the unmigrated cache."""
import numpy as np
import pytest

from oracle import model as om
from oracle import paged
from workloads import configs, gen
from helpers import oracle_weights, shape_of

RNG = np.random.default_rng(7)
L, P, PAGE, HKV, D = 3, 12, 4, 2, 5


def rand_pool():
    return RNG.integers(0, 2**16, size=(L, 2, P, PAGE, HKV, D), dtype=np.uint16)


def test_logical_view_and_pack_brute_force():
    pool = rand_pool()
    bt = RNG.permutation(P)[:8].astype(np.int32)
    n = 29
    lv = paged.logical_view(pool, bt, n)
    for l in range(L):
        for kv in range(2):
            for t in range(n):
                np.testing.assert_array_equal(lv[l, kv, t], pool[l, kv, bt[t // PAGE], t % PAGE])
    for start, cnt in ((0, 29), (3, 9), (12, 4), (27, 2), (5, 0)):
        ch = paged.pack(pool, bt, start, cnt)
        assert ch.shape == (L, 2, cnt, HKV, D)
        for l in range(L):
            for kv in range(2):
                for i in range(cnt):
                    t = start + i
                    np.testing.assert_array_equal(ch[l, kv, i], pool[l, kv, bt[t // PAGE], t % PAGE])


def hdr(start, cnt, req=7, epoch=3, shape=(L, HKV, D, 2)):
    return paged.ChunkHeader(req, epoch, start, cnt, *shape)


def test_assemble_brute_force_and_sentinels():
    src = rand_pool()
    src_bt = RNG.permutation(P)[:8].astype(np.int32)
    dst = np.full((L, 2, P, PAGE, HKV, D), 0x7FA5, dtype=np.uint16)
    free = np.array([1, 4, 5, 8, 9, 11], dtype=np.int32)     # others are occupied
    dst_bt = free[RNG.permutation(len(free))]
    before = dst.copy()
    pieces = [(5, 4), (9, 7), (16, 6)]                        # unaligned starts and ends
    hdrs = [hdr(s, c) for s, c in pieces]
    chunks = [paged.pack(src, src_bt, s, c) for s, c in pieces]
    assert paged.assemble(dst, dst_bt, hdrs, chunks, 7, 3)
    touched = set()
    for s, c in pieces:
        for t in range(s, s + c):
            touched.add((int(dst_bt[t // PAGE]), t % PAGE))
            np.testing.assert_array_equal(dst[:, :, dst_bt[t // PAGE], t % PAGE],
                                          src[:, :, src_bt[t // PAGE], t % PAGE])
    for pg in range(P):
        for sl in range(PAGE):
            if (pg, sl) not in touched:
                np.testing.assert_array_equal(dst[:, :, pg, sl], before[:, :, pg, sl])
    # pack of the assembled range returns the chunks
    for (s, c), ch in zip(pieces, chunks):
        np.testing.assert_array_equal(paged.pack(dst, dst_bt, s, c), ch)


@pytest.mark.parametrize("bad,code", [
    (dict(req=8), "WRONG_REQUEST"),
    (dict(epoch=2), "STALE_EPOCH"),
    (dict(shape=(L, HKV, D + 1, 2)), "INVALID_ARG"),
])
def test_assemble_rejects_whole_call(bad, code):
    dst = rand_pool()
    before = dst.copy()
    bt = np.arange(6, dtype=np.int32)
    good = hdr(0, 4)
    wrong = hdr(4, 4, **bad)
    chunks = [np.zeros((L, 2, 4, HKV, D), np.uint16)] * 2
    with pytest.raises(paged.Rejected) as e:
        paged.assemble(dst, bt, [good, wrong], chunks, 7, 3)
    assert e.value.code == code
    np.testing.assert_array_equal(dst, before)


def test_assemble_rejects_range_and_overlap():
    dst = rand_pool()
    before = dst.copy()
    bt = np.arange(6, dtype=np.int32)                        # capacity 24
    z = np.zeros((L, 2, 8, HKV, D), np.uint16)
    with pytest.raises(paged.Rejected) as e:
        paged.assemble(dst, bt, [hdr(20, 5)], [z], 7, 3)
    assert e.value.code == "OUT_OF_RANGE"
    with pytest.raises(paged.Rejected) as e:
        paged.assemble(dst, bt, [hdr(0, 8), hdr(7, 3)], [z, z], 7, 3)
    assert e.value.code == "COVERAGE"
    np.testing.assert_array_equal(dst, before)


def test_assemble_skips_invalid_page_entries():
    dst = rand_pool()
    before = dst.copy()
    bt = np.array([0, -1, 3, P + 2], dtype=np.int32)
    ch = RNG.integers(0, 2**16, size=(L, 2, 16, HKV, D), dtype=np.uint16)
    assert not paged.assemble(dst, bt, [hdr(0, 16)], [ch], 7, 3)
    np.testing.assert_array_equal(dst[:, :, 0], ch[:, :, 0:4])
    np.testing.assert_array_equal(dst[:, :, 3], ch[:, :, 8:12])
    for pg in (1, 2, 4, 5, 6, 7, 8, 9, 10, 11):
        np.testing.assert_array_equal(dst[:, :, pg], before[:, :, pg])


@pytest.mark.parametrize("prefix,ranges,n,ok", [
    (96, [(96, 32)], 128, True),
    (96, [(96, 16), (112, 16)], 128, True),
    (96, [(112, 16), (96, 16)], 128, True),       # any order
    (96, [(96, 16)], 128, False),                  # gap at the end
    (96, [(100, 28)], 128, False),                 # gap after the prefix
    (96, [(90, 38)], 128, False),                  # overlaps the prefix
    (96, [(96, 20), (112, 16)], 128, False),       # two ranges claim 112..115
    (96, [(96, 40)], 128, False),                  # past n
    (128, [], 128, True),
    (0, [(0, 128)], 128, True),
    (96, [(96, 32), (50, 0)], 128, True),          # empty range is harmless
    (130, [], 128, False),
])
def test_check_coverage(prefix, ranges, n, ok):
    starts = [r[0] for r in ranges]
    lens = [r[1] for r in ranges]
    assert paged.check_coverage(prefix, starts, lens, n) is ok


def test_assembly_reproduces_unmigrated_cache():
    """Target prefix prefill + assembled source suffix equals the cache of a
    run that never migrated, over every position of [0, n)."""
    cfg = configs.TINY
    glob, layers = gen.model_weights(cfg, seed=0)
    g, ls = oracle_weights(glob, layers)
    shp = shape_of(cfg)
    n, p = 128, 96
    ids = gen.token_ids(n, cfg.vocab, seed=0).tolist()
    shape = (cfg.n_layers, 2, 64, 16, cfg.n_kv_heads, cfg.head_dim)
    src = np.zeros(shape)
    src_bt = gen.block_table(8, 64, 8, 0, 1)
    Kf, Vf, _ = om.prefill(ids, g, ls, shp)
    paged.write_cache(src, src_bt, Kf, Vf)
    dst = np.full(shape, np.nan)
    dst_bt = gen.block_table(8, 64, 8, 0, 2)
    Kp, Vp, _ = om.prefill(ids[:p], g, ls, shp)
    paged.write_cache(dst, dst_bt, Kp, Vp)
    chunks, hdrs = [], []
    for s in range(p, n, 8):
        chunks.append(paged.pack(src, src_bt, s, 8))
        hdrs.append(paged.ChunkHeader(1, 1, s, 8, cfg.n_layers, cfg.n_kv_heads, cfg.head_dim, 8))
    assert paged.check_coverage(p, [h.start_pos for h in hdrs], [h.num_tokens for h in hdrs], n)
    assert paged.assemble(dst, dst_bt, hdrs, chunks, 1, 1)
    lv_dst = paged.logical_view(dst, dst_bt, n)
    lv_src = paged.logical_view(src, src_bt, n)
    np.testing.assert_array_equal(lv_dst[:, :, p:], lv_src[:, :, p:])
    np.testing.assert_allclose(lv_dst[:, :, :p], lv_src[:, :, :p], rtol=1e-9, atol=1e-12)
