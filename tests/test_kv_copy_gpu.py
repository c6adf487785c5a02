"""GPU parity of suffix-block extraction (pack) and assembly against the
oracle: bit-exact on every element, including untouched pages and slots.

Cases: a tiny pool with ragged, unaligned and empty chunks; page sizes 4,
8 and 32 (shorter and longer than a 16-position work unit); the 64-layer /
8-KV-head / d=128 stress layout (8192-token source in shuffled pages, a
1024-page target half occupied by sentinel pages, suffixes of 64, 256, 1024
and 4096 tokens in 32-token chunks); invalid table entries; rejected calls."""
import numpy as np
import pytest
import torch

from helpers import bits, ensure_lib
from oracle import paged
from workloads import configs, gen

pytestmark = pytest.mark.gpu
DEV = "cuda"


@pytest.fixture(scope="module")
def P():
    return ensure_lib()


def chunk_layout(pieces, L, hkv, d):
    """Consecutive arena offsets for (start, count) pieces."""
    out, off = [], 0
    for s, c in pieces:
        out.append((s, c, off))
        off += c * 2 * L * hkv * d * 2
    return out, off


def run_pack_assemble(P, src, src_bt, dst, dst_bt, pieces, req=1, epoch=1):
    L, _, _, _, hkv, d = src.shape
    lay, nbytes = chunk_layout(pieces, L, hkv, d)
    arena = torch.empty(max(nbytes, 16), dtype=torch.uint8, device=DEV)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    descs = [P.ChunkDesc(s, c, off) for s, c, off in lay]
    P.pallas_pack_suffix_blocks(src, src_bt, descs, arena, err)
    hdrs = [P.ChunkHeader(req, epoch, s, c, off, L, hkv, d, 2) for s, c, off in lay]
    P.pallas_assemble_kv(dst, dst_bt, hdrs, arena, req, epoch, err)
    torch.cuda.synchronize()
    return arena, lay, int(err.item())


def arena_chunk(arena, off, c, L, hkv, d):
    n = c * 2 * L * hkv * d * 2
    return arena[off:off + n].cpu().numpy().view(np.uint16).reshape(L, 2, c, hkv, d)


def test_tiny_ragged_chunks(P):
    L, Pg, hkv, d = 2, 64, 2, 64
    src = gen.kv_pool_normal(L, Pg, 16, hkv, d, seed=11)
    src_bt = torch.from_numpy(gen.block_table(8, Pg, 8, 11, 1))
    dst = torch.full((L, 2, Pg, 16, hkv, d), 0, dtype=torch.int16).view(torch.bfloat16)
    dst.view(torch.int16).fill_(gen.SENTINEL_BITS)
    dst_bt = torch.from_numpy(gen.block_table(8, Pg, 8, 11, 2))
    pieces = [(96, 5), (101, 0), (101, 11), (112, 16), (0, 3), (3, 1)]
    src_np, dst_np = bits(src), bits(dst)
    arena, lay, err = run_pack_assemble(P, src.to(DEV), src_bt.to(DEV), dst_gpu := dst.to(DEV),
                                        dst_bt.to(DEV), pieces)
    assert err == 0
    hdrs = []
    for s, c, off in lay:
        want = paged.pack(src_np, src_bt.numpy(), s, c)
        np.testing.assert_array_equal(arena_chunk(arena, off, c, L, hkv, d), want)
        hdrs.append(paged.ChunkHeader(1, 1, s, c, L, hkv, d, 2))
    chunks = [paged.pack(src_np, src_bt.numpy(), s, c) for s, c, _ in lay]
    assert paged.assemble(dst_np, dst_bt.numpy(), hdrs, chunks, 1, 1)
    np.testing.assert_array_equal(bits(dst_gpu), dst_np)


@pytest.mark.parametrize("page", [4, 8, 32])
def test_other_page_sizes_bit_exact(P, page):
    """Pages shorter than a 16-position run (each position looks up its own
    page) and longer ones (a run spans at most two pages), with unaligned
    and ragged chunks."""
    L, hkv, d = 2, 2, 64
    n_src = 8 * 32
    pages = n_src // page
    src = gen.kv_pool_normal(L, pages, page, hkv, d, seed=12)
    src_bt = torch.from_numpy(gen.block_table(pages, pages, pages, 12, 1))
    dst_pages = 2 * pages
    dst = torch.empty((L, 2, dst_pages, page, hkv, d), dtype=torch.bfloat16)
    dst.view(torch.int16).fill_(gen.SENTINEL_BITS)
    dst_bt = torch.from_numpy(gen.block_table(pages, dst_pages, pages, 12, 2))
    pieces = [(3, 29), (32, 1), (33, 70), (103, 16), (119, n_src - 119)]
    src_np, dst_np = bits(src), bits(dst)
    arena, lay, err = run_pack_assemble(P, src.to(DEV), src_bt.to(DEV), dst_gpu := dst.to(DEV),
                                        dst_bt.to(DEV), pieces)
    assert err == 0
    hdrs, chunks = [], []
    for s0, c, off in lay:
        want = paged.pack(src_np, src_bt.numpy(), s0, c)
        np.testing.assert_array_equal(arena_chunk(arena, off, c, L, hkv, d), want)
        hdrs.append(paged.ChunkHeader(1, 1, s0, c, L, hkv, d, 2))
        chunks.append(want)
    assert paged.assemble(dst_np, dst_bt.numpy(), hdrs, chunks, 1, 1)
    np.testing.assert_array_equal(bits(dst_gpu), dst_np)


@pytest.mark.parametrize("s", configs.STRESS_SUFFIXES)
def test_stress_layout_bit_exact(P, s):
    cfg = configs.STRESS_KV
    L, hkv, d = cfg.n_layers, cfg.n_kv_heads, cfg.head_dim
    n_src = configs.STRESS_SOURCE_TOKENS
    src_pages = n_src // 16
    src = gen.kv_pool_normal(L, src_pages, 16, hkv, d, seed=4, device=DEV)
    src_bt = torch.from_numpy(gen.block_table(src_pages, src_pages, src_pages, 4, 1)).to(DEV)
    tp = configs.STRESS_TARGET_PAGES
    occupied = np.sort(gen.permutation(tp, 4, 2)[: tp // 2])
    free = np.setdiff1d(np.arange(tp), occupied).astype(np.int32)
    dst = torch.empty((L, 2, tp, 16, hkv, d), dtype=torch.bfloat16, device=DEV)
    dst.view(torch.int16).fill_(gen.SENTINEL_BITS)
    dst_bt = torch.from_numpy(gen.block_table(src_pages, tp, src_pages, 4, 3,
                                              free_pages=free)).to(DEV)
    start = n_src - s
    pieces = [(t, min(configs.STRESS_CHUNK, n_src - t)) for t in range(start, n_src, configs.STRESS_CHUNK)]
    arena, lay, err = run_pack_assemble(P, src, src_bt, dst, dst_bt, pieces)
    assert err == 0
    src_np = bits(src)
    sbt, dbt = src_bt.cpu().numpy(), dst_bt.cpu().numpy()
    # every chunk equals the oracle's extraction
    for s0, c, off in lay:
        np.testing.assert_array_equal(arena_chunk(arena, off, c, L, hkv, d),
                                      paged.pack(src_np, sbt, s0, c))
    dst_np = bits(dst)
    # assembled suffix equals the source's logical view
    np.testing.assert_array_equal(paged.logical_view(dst_np, dbt, n_src)[:, :, start:],
                                  paged.logical_view(src_np, sbt, n_src)[:, :, start:])
    # occupied pages keep their sentinels; so do target slots before the suffix
    assert np.all(dst_np[:, :, occupied] == gen.SENTINEL_BITS)
    untouched = paged.logical_view(dst_np, dbt, start)
    assert np.all(untouched == gen.SENTINEL_BITS)


def test_invalid_table_entries_skip_and_flag(P):
    L, Pg, hkv, d = 2, 16, 2, 64
    src = gen.kv_pool_normal(L, Pg, 16, hkv, d, seed=5, device=DEV)
    src_bt = torch.arange(4, dtype=torch.int32, device=DEV)
    dst = torch.zeros((L, 2, Pg, 16, hkv, d), dtype=torch.bfloat16, device=DEV)
    dst_bt = torch.tensor([2, -1, 7, Pg + 5], dtype=torch.int32, device=DEV)
    arena, lay, err = run_pack_assemble(P, src, src_bt, dst, dst_bt, [(0, 64)])
    assert err & 1
    sn, dn = bits(src), bits(dst)
    np.testing.assert_array_equal(dn[:, :, 2], sn[:, :, 0])
    np.testing.assert_array_equal(dn[:, :, 7], sn[:, :, 2])
    others = [p for p in range(Pg) if p not in (2, 7)]
    assert np.all(dn[:, :, others] == 0)


@pytest.mark.parametrize("bad", ["epoch", "request", "overlap"])
def test_rejected_assembly_writes_nothing(P, bad):
    L, Pg, hkv, d = 2, 16, 2, 64
    dst = gen.kv_pool_normal(L, Pg, 16, hkv, d, seed=6, device=DEV)
    before = bits(dst)
    arena = torch.ones(64 * 2 * L * hkv * d * 2, dtype=torch.uint8, device=DEV)
    bt = torch.arange(4, dtype=torch.int32, device=DEV)
    row = 2 * L * hkv * d * 2
    h1 = P.ChunkHeader(9, 2, 0, 32, 0, L, hkv, d, 2)
    h2 = {"epoch": P.ChunkHeader(9, 1, 32, 32, 32 * row, L, hkv, d, 2),
          "request": P.ChunkHeader(8, 2, 32, 32, 32 * row, L, hkv, d, 2),
          "overlap": P.ChunkHeader(9, 2, 31, 32, 32 * row, L, hkv, d, 2)}[bad]
    with pytest.raises(P.PallasError):
        P.pallas_assemble_kv(dst, bt, [h1, h2], arena, 9, 2)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(bits(dst), before)
