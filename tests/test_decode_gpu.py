"""GPU parity of the decode step at the large decoder's layer shape (2
layers, hidden 5120, 64/8 heads, ffn 25600) against the oracle's decode over
the oracle's cache: one sequence and a batch of three, logits within
max|gpu - ref| <= 1e-2 max|ref| per row.  At this shape the O and down
projections split K three ways over workgroups and reduce the partial sums
in the last workgroup of each tile (Q|K|V, gate|up and lm_head stream whole
tiles); two identical calls give identical logits.  Also a token decoding
at position 0 (an empty cache) in one batch with another sequence, and a
batch of eight at the large attention shape whose positions span the
decode attention's key splits."""
import numpy as np
import pytest
import torch

from helpers import TOL, empty_pool, ensure_lib, gpu_model, kv_logical, oracle_weights, rel_err, shape_of
from oracle import model as om
from workloads import configs, gen

pytestmark = pytest.mark.gpu
DEV = "cuda"


@pytest.fixture(scope="module")
def P():
    return ensure_lib()


def test_decode_large_layer_shape(P):
    cfg = configs.LARGE.replace(n_layers=2, vocab=4096, name="large-L2")
    glob, layers = gen.model_weights(cfg, seed=31, gain_sigma=0.1)
    model = gpu_model(P, cfg, glob, layers)
    lens = [40, 17, 63]
    ids = [gen.token_ids(n + 1, cfg.vocab, seed=31, stream=i).numpy() for i, n in enumerate(lens)]
    pages = [(n + 1 + 15) // 16 for n in lens]
    tables = gen.disjoint_block_tables(pages, 16, 5, 31, 1)
    d_bt = torch.tensor(tables, dtype=torch.int32, device=DEV)
    pool = empty_pool(cfg, 16, fill_bits=0)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    ws = model.workspace(max(lens), 3)
    for i, n in enumerate(lens):
        model.prefill_prefix(torch.tensor(ids[i][:n], dtype=torch.int32, device=DEV), [0, n], d_bt[i:i + 1],
                             pool, ws, err)
    torch.cuda.synchronize()
    snapshot = pool.clone()
    toks = torch.tensor([x[n] for x, n in zip(ids, lens)], dtype=torch.int32, device=DEV)
    one = torch.empty((1, cfg.vocab), dtype=torch.float32, device=DEV)
    model.decode_step(toks[:1], lens[:1], d_bt[:1], pool, one, ws, err)
    pool.copy_(snapshot)
    batch = torch.empty((3, cfg.vocab), dtype=torch.float32, device=DEV)
    model.decode_step(toks, lens, d_bt, pool, batch, ws, err)
    pool.copy_(snapshot)
    again = torch.empty_like(batch)
    model.decode_step(toks, lens, d_bt, pool, again, ws, err)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    assert torch.equal(batch, again)
    g, ls = oracle_weights(glob, layers)
    shp = shape_of(cfg)
    for i, n in enumerate(lens):
        K, V, _ = om.prefill(list(ids[i][:n]), g, ls, shp)
        ref, _, _ = om.decode(int(ids[i][n]), n, K, V, g, ls, shp)
        e = rel_err(batch[i].cpu().double().numpy(), ref)
        assert e <= TOL, f"sequence {i}: logits rel err {e:.3g}"
        if i == 0:
            assert rel_err(one[0].cpu().double().numpy(), ref) <= TOL


def test_decode_at_position_zero_in_a_batch(P):
    """The degenerate context: a token at position 0 over an empty cache
    attends only to itself.  It decodes in one batch with a sequence at
    position 20.  Both rows of logits and the K/V each step writes into
    its slot are checked against the oracle's decode."""
    cfg = configs.TINY.replace(qk_norm=True)
    glob, layers = gen.model_weights(cfg, seed=32, gain_sigma=0.1)
    model = gpu_model(P, cfg, glob, layers)
    lens = [0, 20]
    ids = [gen.token_ids(n + 1, cfg.vocab, seed=32, stream=i).numpy() for i, n in enumerate(lens)]
    pages = [(n + 1 + 15) // 16 for n in lens]
    tables = gen.disjoint_block_tables(pages, 8, 2, 32, 1)
    d_bt = torch.tensor(tables, dtype=torch.int32, device=DEV)
    pool = empty_pool(cfg, 8, fill_bits=0)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    ws = model.workspace(32, 2)
    model.prefill_prefix(torch.tensor(ids[1][:20], dtype=torch.int32, device=DEV), [0, 20], d_bt[1:2], pool,
                         ws, err)
    toks = torch.tensor([x[n] for x, n in zip(ids, lens)], dtype=torch.int32, device=DEV)
    logits = torch.empty((2, cfg.vocab), dtype=torch.float32, device=DEV)
    model.decode_step(toks, lens, d_bt, pool, logits, ws, err)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    g, ls = oracle_weights(glob, layers)
    shp = shape_of(cfg)
    empty = [np.zeros((0, cfg.n_kv_heads, cfg.head_dim))] * cfg.n_layers
    for i, n in enumerate(lens):
        if n:
            K, V, _ = om.prefill(list(ids[i][:n]), g, ls, shp)
        else:
            K, V = empty, empty
        ref, k_new, v_new = om.decode(int(ids[i][n]), n, K, V, g, ls, shp)
        e = rel_err(logits[i].cpu().double().numpy(), ref)
        assert e <= TOL, f"sequence {i} at position {n}: logits rel err {e:.3g}"
        lv = kv_logical(pool, tables[i], n + 1)
        for l in range(cfg.n_layers):
            assert rel_err(lv[l, 0, n], k_new[l][0]) <= TOL
            assert rel_err(lv[l, 1, n], v_new[l][0]) <= TOL


def test_decode_large_heads_batch_of_eight(P):
    """Eight sequences decoding in one call at the large model's attention
    shape (64 query heads over 8 KV heads, head_dim 128, QK-norm; a narrower
    residual stream and FFN keep the oracle cheap), at positions 0 (empty
    cache), 1, 63, 64, 65 (one and two 64-key splits), 200, 1023 and 1100
    (16 and 18 splits: the combine reads its records in batches of 16)."""
    cfg = configs.LARGE.replace(n_layers=2, vocab=4096, hidden=1024, ffn=4096, name="large-heads-L2")
    glob, layers = gen.model_weights(cfg, seed=33, gain_sigma=0.1)
    model = gpu_model(P, cfg, glob, layers)
    lens = [0, 1, 63, 64, 65, 200, 1023, 1100]
    ids = [gen.token_ids(n + 1, cfg.vocab, seed=33, stream=i).numpy() for i, n in enumerate(lens)]
    pages = [(n + 1 + 15) // 16 for n in lens]
    tables = gen.disjoint_block_tables(pages, 200, 70, 33, 1)
    d_bt = torch.tensor(tables, dtype=torch.int32, device=DEV)
    pool = empty_pool(cfg, 200, fill_bits=0)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    ws = model.workspace(max(lens), 8)
    for i, n in enumerate(lens):
        if n:
            model.prefill_prefix(torch.tensor(ids[i][:n], dtype=torch.int32, device=DEV), [0, n], d_bt[i:i + 1],
                                 pool, ws, err)
    toks = torch.tensor([x[n] for x, n in zip(ids, lens)], dtype=torch.int32, device=DEV)
    logits = torch.empty((8, cfg.vocab), dtype=torch.float32, device=DEV)
    model.decode_step(toks, lens, d_bt, pool, logits, ws, err)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    g, ls = oracle_weights(glob, layers)
    shp = shape_of(cfg)
    for i, n in enumerate(lens):
        if n:
            K, V, _ = om.prefill(list(ids[i][:n]), g, ls, shp)
        else:
            K = V = [np.zeros((0, cfg.n_kv_heads, cfg.head_dim)) for _ in range(cfg.n_layers)]
        ref, _, _ = om.decode(int(ids[i][n]), n, K, V, g, ls, shp)
        e = rel_err(logits[i].cpu().double().numpy(), ref)
        assert e <= TOL, f"sequence {i} at position {n}: logits rel err {e:.3g}"
