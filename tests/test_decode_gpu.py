"""GPU parity of the decode step at the large decoder's layer shape (2
layers, hidden 5120, 64/8 heads, ffn 25600) against the oracle's decode over
the oracle's cache: one sequence and a batch of three, logits within
max|gpu - ref| <= 1e-2 max|ref| per row.  At this shape the skinny
projections split K over workgroups (Q|K|V and gate|up two ways, O and down
four ways) and reduce the partial sums in the last workgroup of each tile;
two identical calls give identical logits."""
import numpy as np
import pytest
import torch

from helpers import TOL, empty_pool, ensure_lib, gpu_model, oracle_weights, rel_err, shape_of
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
