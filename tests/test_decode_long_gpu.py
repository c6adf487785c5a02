"""Decode parity against the oracle at long contexts and full vocabulary.

From position 1024 on, decode attention runs more than 16 splits of 64 keys
and its combine pass reads the split records in several batches of 16;
from 4000 on, more than 62.  The lm_head of the 151936-token vocabulary has
9496 weight tiles.  Logits within max|gpu - ref| <= 1e-2 max|ref| per row.

* Tiny decoder (2 layers, vocab 151936), the oracle end to end: it prefills
  its own cache of 8000 tokens and decodes at positions 1100, 4000 and 8000;
  the GPU prefills three sequences of those lengths into their own tables
  and decodes all three in one batch.
* The large decoder's layer shape (2 layers, hidden 5120, 64/8 heads, ffn
  25600, vocab 151936) at the same positions.  The oracle cannot prefill
  13,100 tokens at this shape in test time, so the cache is checked layer
  by layer (layer 0 from the embedding, layer 1 from the GPU's input to it,
  and layer 0's residual update on each sequence's last 64 rows, whose
  attention reads up to 8000 keys), and the oracle's decode then runs over
  the GPU's cache.
* The concurrent workload at reduced depth: 2 layers of the mid decoder
  (vocab 151936), the workload's 8 context lengths (1000-8000) and prefix
  fractions, suffixes streamed in 32-token chunks and assembled; the cache
  checked layer by layer as above, then the 8-request batched decode over
  the assembled caches against the oracle's decode over them."""
import numpy as np
import pytest
import torch

from helpers import (TOL, check_layer_local, empty_pool, ensure_lib, gpu_model, kv_logical,
                     oracle_weights, rel_err, residual_rows, shape_of, to_np64)
from oracle import model as om
from recon import Recon
from workloads import configs, gen

pytestmark = [pytest.mark.gpu, pytest.mark.slow]
DEV = "cuda"
LENS = [1100, 4000, 8000]


@pytest.fixture(scope="module")
def P():
    return ensure_lib()


def prefill_three(P, cfg, glob, layers, ids, seed):
    """GPU prefill of ids[:n] for n in LENS (varlen, one table each, with
    room for slot n), then one batched decode of ids[n] at position n."""
    model = gpu_model(P, cfg, glob, layers)
    pages = [(n + 1 + 15) // 16 for n in LENS]
    tables = gen.disjoint_block_tables(pages, sum(pages), max(pages), seed, 1)
    d_bt = torch.tensor(tables, dtype=torch.int32, device=DEV)
    pool = empty_pool(cfg, sum(pages), fill_bits=0)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    cu = np.cumsum([0] + LENS).tolist()
    d_ids = torch.tensor(np.concatenate([ids[:n] for n in LENS]), dtype=torch.int32, device=DEV)
    ws = model.workspace(cu[-1], len(LENS))
    model.prefill_prefix(d_ids, cu, d_bt, pool, ws, err)
    torch.cuda.synchronize()
    r1 = residual_rows(ws, cu[-1], cfg.hidden).double().cpu().numpy()   # layer 1's input
    del ws
    toks = torch.tensor([ids[n] for n in LENS], dtype=torch.int32, device=DEV)
    logits = torch.empty((len(LENS), cfg.vocab), dtype=torch.float32, device=DEV)
    wsd = model.workspace(len(LENS), len(LENS))
    model.decode_step(toks, LENS, d_bt, pool, logits, wsd, err)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    return tables, pool, cu, r1, logits.double().cpu().numpy()


def test_tiny_long_positions_full_vocab(P):
    cfg = configs.TINY.replace(vocab=151936, qk_norm=True, name="tiny-v151936")
    glob, layers = gen.model_weights(cfg, seed=41, gain_sigma=0.1)
    ids = gen.token_ids(max(LENS) + 1, cfg.vocab, seed=41).numpy()
    tables, pool, cu, _, logits = prefill_three(P, cfg, glob, layers, ids, 41)
    g, ls = oracle_weights(glob, layers)
    shp = shape_of(cfg)
    K, V, _ = om.prefill(list(ids[:max(LENS)]), g, ls, shp)
    for i, n in enumerate(LENS):
        lv = kv_logical(pool, tables[i], n)
        for l in range(cfg.n_layers):
            for kv, ref in ((0, K[l][:n]), (1, V[l][:n])):
                e = rel_err(lv[l, kv], ref)
                assert e <= TOL, f"sequence {i} layer {l} {'KV'[kv]}: {e:.3g}"
        ref, _, _ = om.decode(int(ids[n]), n, [k[:n] for k in K], [v[:n] for v in V], g, ls, shp)
        e = rel_err(logits[i], ref)
        print(f"position {n}: logits rel err {e:.2e}")
        assert e <= TOL, f"position {n}: logits {e:.3g}"


def test_large_layer_shape_long_positions(P):
    cfg = configs.LARGE.replace(n_layers=2, name="large-L2")
    glob, layers = gen.model_weights(cfg, seed=42, gain_sigma=0.1, device=DEV)
    ids = gen.token_ids(max(LENS) + 1, cfg.vocab, seed=42).numpy()
    tables, pool, cu, r1, logits = prefill_three(P, cfg, glob, layers, ids, 42)
    shp = shape_of(cfg)
    ws = [{k: to_np64(v) for k, v in l.items()} for l in layers]
    rows = np.concatenate([ids[:n] for n in LENS])
    r0 = to_np64(glob["embed"][torch.as_tensor(rows, dtype=torch.long, device=DEV)])
    caches = [kv_logical(pool, tables[i], n) for i, n in enumerate(LENS)]
    check_layer_local(r0, cu, ws[0], shp, [c[0, 0] for c in caches], [c[0, 1] for c in caches],
                      r_next=r1, tail=64, label="layer 0")
    check_layer_local(r1, cu, ws[1], shp, [c[1, 0] for c in caches], [c[1, 1] for c in caches],
                      label="layer 1")
    toks = [int(ids[n]) for n in LENS]
    # The oracle embeds by row lookup: give it the three decode tokens' rows.
    g = {"embed": to_np64(glob["embed"][torch.as_tensor(toks, device=DEV)]),
         "final_norm": to_np64(glob["final_norm"]), "lm_head": to_np64(glob["lm_head"])}
    for i, n in enumerate(LENS):
        ref, _, _ = om.decode(i, n, [caches[i][l, 0] for l in range(2)], [caches[i][l, 1] for l in range(2)],
                              g, ws, shp)
        e = rel_err(logits[i], ref)
        print(f"position {n}: logits rel err {e:.2e}")
        assert e <= TOL, f"position {n}: logits {e:.3g}"


def test_concurrent_reduced_depth_batched_decode(P):
    full = configs.workload("concurrent")
    from workloads.configs import Workload
    wl = Workload("concurrent-L2", full.model.with_layers(2), full.ctx, full.prefix, full.chunk_tokens)
    r = Recon(P, wl)
    r.check_properties()
    r.check_prefill_layer(0, tail=64)
    r.check_prefill_layer(1)
    toks = r.tokens.cpu().numpy().tolist()
    g = {"embed": to_np64(r.glob["embed"][r.tokens.long()]),
         "final_norm": to_np64(r.glob["final_norm"]), "lm_head": to_np64(r.glob["lm_head"])}
    ws = [r.lazy[0], {k: to_np64(v) for k, v in r.layers[1].items()}]
    for i, n in enumerate(r.ns):
        c = r.kv(r.dst, r.dst_tab, i, n, 0), r.kv(r.dst, r.dst_tab, i, n, 1)
        ref, _, _ = om.decode(i, n, [c[0][0], c[1][0]], [c[0][1], c[1][1]], g, ws, r.shp)
        e = rel_err(r.logits_dst[i].double().cpu().numpy(), ref)
        print(f"request {i} at position {n} (token {toks[i]}): logits rel err {e:.2e}")
        assert e <= TOL, f"request {i}: logits {e:.3g}"
