"""End-to-end reconstruction on the GPU against the oracle's unmigrated run:
source full prefill -> pack the suffix -> target prefix prefill -> assemble
-> decode one token at position n.

Checks: the assembled cache equals the source's on the suffix bit for bit
and the oracle's cache within tolerance on the prefix (assembly equals the
unmigrated cache); decode logits equal the oracle's decode over the
oracle's unmigrated cache within tolerance; a batched decode over several
assembled requests."""
import numpy as np
import pytest
import torch

from helpers import (TOL, empty_pool, ensure_lib, gpu_model, kv_logical, oracle_weights,
                     rel_err, shape_of)
from oracle import model as om
from oracle import paged
from workloads import configs, gen

pytestmark = pytest.mark.gpu
DEV = "cuda"


@pytest.fixture(scope="module")
def P():
    return ensure_lib()


def reconstruct(P, model, cfg, reqs, src_pages, dst_pages, chunk=None, seed=0):
    """reqs: list of (ids[n+1], p).  Returns target pool, target tables,
    source pool, source tables and decode logits (one row per request)."""
    B = len(reqs)
    ns = [len(ids) - 1 for ids, _ in reqs]
    max_pages = max((n + 1 + 15) // 16 for n in ns)
    src_tab = gen.disjoint_block_tables([(n + 15) // 16 for n in ns], src_pages, max_pages, seed, 1)
    dst_tab = gen.disjoint_block_tables([(n + 1 + 15) // 16 for n in ns], dst_pages, max_pages, seed, 2)
    src = empty_pool(cfg, src_pages, fill_bits=0)
    dst = empty_pool(cfg, dst_pages, fill_bits=0x7FA5)
    d_src_tab = torch.tensor(src_tab, dtype=torch.int32, device=DEV)
    d_dst_tab = torch.tensor(dst_tab, dtype=torch.int32, device=DEV)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    row = 2 * cfg.n_layers * cfg.n_kv_heads * cfg.head_dim * 2
    for i, (ids, p) in enumerate(reqs):
        n = ns[i]
        # source: full prefill of [0, n) (the unmigrated cache)
        ws = model.workspace(n)
        model.prefill_prefix(torch.tensor(ids[:n], dtype=torch.int32, device=DEV), [0, n],
                             d_src_tab[i:i + 1], src, ws, err)
        # pack [p, n) in chunks
        step = chunk or (n - p)
        pieces = [(t, min(step, n - t)) for t in range(p, n, step)]
        offs = np.cumsum([0] + [c * row for _, c in pieces])
        arena = torch.empty(max(int(offs[-1]), 16), dtype=torch.uint8, device=DEV)
        P.pallas_pack_suffix_blocks(src, d_src_tab[i], [P.ChunkDesc(s, c, int(o)) for (s, c), o in
                                                        zip(pieces, offs)], arena, err)
        # target: prefix prefill, then assembly
        ws2 = model.workspace(p)
        model.prefill_prefix(torch.tensor(ids[:p], dtype=torch.int32, device=DEV), [0, p],
                             d_dst_tab[i:i + 1], dst, ws2, err)
        hdrs = [P.ChunkHeader(100 + i, 7, s, c, int(o), cfg.n_layers, cfg.n_kv_heads, cfg.head_dim, 2)
                for (s, c), o in zip(pieces, offs)]
        assert P.pallas_check_coverage(p, [h.start_pos for h in hdrs], [h.num_tokens for h in hdrs], n) == 0
        P.pallas_assemble_kv(dst, d_dst_tab[i], hdrs, arena, 100 + i, 7, err)
        torch.cuda.synchronize()
    toks = torch.tensor([ids[n] for (ids, _), n in zip(reqs, ns)], dtype=torch.int32, device=DEV)
    logits = torch.empty((B, cfg.vocab), dtype=torch.float32, device=DEV)
    ws = model.workspace(B, B)
    model.decode_step(toks, ns, d_dst_tab, dst, logits, ws, err)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    return dst, dst_tab, src, src_tab, logits.cpu().numpy().astype(np.float64)


def check(cfg, glob, layers, reqs, dst, dst_tab, src, src_tab, logits):
    g, ls = oracle_weights(glob, layers)
    shp = shape_of(cfg)
    for i, (ids, p) in enumerate(reqs):
        n = len(ids) - 1
        lv_dst = kv_logical(dst, dst_tab[i], n)
        lv_src = kv_logical(src, src_tab[i], n)
        # suffix: bit-exact copy of the source cache
        np.testing.assert_array_equal(lv_dst[:, :, p:], lv_src[:, :, p:])
        K, V, _ = om.prefill(list(ids[:n]), g, ls, shp)
        for l in range(cfg.n_layers):
            for kv, ref in ((0, K[l]), (1, V[l])):
                assert rel_err(lv_dst[l, kv], ref) <= TOL, (i, l, kv)
        ref_logits, _, _ = om.decode(int(ids[n]), n, K, V, g, ls, shp)
        e = rel_err(logits[i], ref_logits)
        assert e <= TOL, f"request {i}: logits rel err {e:.3g}"
        # the new token's K/V went to slot n
        lv_new = kv_logical(dst, dst_tab[i], n + 1)[:, :, n]
        assert np.all(np.isfinite(lv_new))


@pytest.mark.parametrize("qk_norm", [False, True])
def test_tiny_reconstruction(P, qk_norm):
    cfg = configs.TINY.replace(qk_norm=qk_norm)
    glob, layers = gen.model_weights(cfg, seed=0, gain_sigma=0.1 if qk_norm else None)
    model = gpu_model(P, cfg, glob, layers)
    ids = gen.token_ids(129, cfg.vocab, seed=0).numpy()
    reqs = [(ids, 96)]
    out = reconstruct(P, model, cfg, reqs, 64, 64)
    check(cfg, glob, layers, reqs, *out)


def test_unaligned_split_chunked(P):
    """Split inside a page (the large workload's 3000 = 187*16 + 8 case) and
    a suffix streamed in 32-token chunks."""
    cfg = configs.MID.replace(n_layers=2, vocab=4096, name="mid-L2")
    glob, layers = gen.model_weights(cfg, seed=4, gain_sigma=0.1)
    model = gpu_model(P, cfg, glob, layers)
    ids = gen.token_ids(301, cfg.vocab, seed=4).numpy()
    reqs = [(ids, 200)]
    out = reconstruct(P, model, cfg, reqs, 40, 40, chunk=32, seed=4)
    check(cfg, glob, layers, reqs, *out)


def test_batched_decode_over_several_requests(P):
    cfg = configs.MID.replace(n_layers=2, vocab=4096, name="mid-L2")
    glob, layers = gen.model_weights(cfg, seed=5, gain_sigma=0.1)
    model = gpu_model(P, cfg, glob, layers)
    reqs = []
    for i, (n, p) in enumerate([(150, 96), (64, 48), (233, 160)]):
        reqs.append((gen.token_ids(n + 1, cfg.vocab, seed=5, stream=i).numpy(), p))
    out = reconstruct(P, model, cfg, reqs, 48, 48, chunk=32, seed=5)
    check(cfg, glob, layers, reqs, *out)
