"""GPU parity of chunked prefill (a prefix prefilled chunk by chunk, each
chunk attending to the earlier chunks' K/V through the pool) against the
oracle's whole-prefix prefill, within max|gpu - ref| <= 1e-2 max|ref| per
(layer, K|V) over the written positions.

Shapes: the tiny decoder at full depth with ragged chunks whose starts are
not multiples of 16 or 32 (a chunk of one token among them); the mid
decoder's layer shape in 256-token chunks with a ragged tail; several
sequences at different start positions in one call; chunks of more than
256 rows starting at multiples of 32, which must give the bytes of one
prefill over the whole prefix."""
import numpy as np
import pytest
import torch

from helpers import (TOL, check_layer_local, empty_pool, ensure_lib, gpu_model, kv_logical,
                     oracle_weights, rel_err, residual_rows, shape_of)
from oracle import model as om
from workloads import configs, gen

pytestmark = pytest.mark.gpu
DEV = "cuda"


@pytest.fixture(scope="module")
def P():
    return ensure_lib()


def chunked(model, cfg, ids, bounds, bt, pool, err):
    """Prefill ids[a:b) for each (a, b) in order, one call per chunk.
    Returns the residual each call fed its last layer, [n, H] float64 over
    the chunks' rows (the workspace's residual section after each call)."""
    d_bt = torch.tensor(np.asarray(bt)[None], dtype=torch.int32, device=DEV)
    ws = model.workspace(max(b - a for a, b in bounds))
    rows = []
    for a, b in bounds:
        model.prefill_chunk(torch.tensor(ids[a:b], dtype=torch.int32, device=DEV), [0, b - a], [a],
                            d_bt, pool, ws, err)
        torch.cuda.synchronize()
        rows.append(residual_rows(ws, b - a, cfg.hidden).double().cpu().numpy())
    return np.concatenate(rows)


def check(cfg, glob, layers, ids, pool, bt, n_layers=None):
    """End-to-end oracle parity per (layer, K|V)."""
    g, ls = oracle_weights(glob, layers)
    L = cfg.n_layers if n_layers is None else n_layers
    shp = shape_of(cfg)
    K, V, _ = om.prefill(list(ids), g, ls, shp, n_layers=L)
    lv = kv_logical(pool, bt, len(ids))
    for l in range(L):
        for kv, ref in ((0, K[l]), (1, V[l])):
            e = rel_err(lv[l, kv], ref)
            assert e <= TOL, f"layer {l} {'KV'[kv]}: rel err {e:.3g}"


def check_two_layers(cfg, glob, layers, ids, pool, bt, r1, tail, label):
    """Layer-local oracle parity of a 2-layer model's prefill: layer 0 from
    the embedding (the oracle's own input), with its residual update on the
    last ``tail`` rows; layer 1 from ``r1``, the GPU's input to it.  Also
    prints layer 1's error against the end-to-end oracle, which adds the
    effect of layer 0's bf16 rounding differences on layer 1's input."""
    g, ls = oracle_weights(glob, layers)
    shp = shape_of(cfg)
    n = len(ids)
    lv = kv_logical(pool, bt, n)
    r0 = g["embed"][np.asarray(ids, dtype=np.int64)]
    w0 = check_layer_local(r0, [0, n], ls[0], shp, [lv[0, 0]], [lv[0, 1]], r_next=r1, tail=tail,
                           label=f"{label} layer 0")
    w1 = check_layer_local(r1, [0, n], ls[1], shp, [lv[1, 0]], [lv[1, 1]], label=f"{label} layer 1")
    K, V, _ = om.prefill(list(ids), g, ls, shp)
    e2e = (rel_err(lv[1, 0], K[1]), rel_err(lv[1, 1], V[1]))
    print(f"{label}: layer 0 K {w0[0]:.2e} V {w0[1]:.2e} update {w0[2]:.2e}; layer 1 layer-local "
          f"K {w1[0]:.2e} V {w1[1]:.2e}; layer 1 end to end K {e2e[0]:.2e} V {e2e[1]:.2e}")


@pytest.mark.parametrize("qk_norm", [False, True])
def test_tiny_ragged_chunks(P, qk_norm):
    cfg = configs.TINY.replace(qk_norm=qk_norm)
    glob, layers = gen.model_weights(cfg, seed=4, gain_sigma=0.1 if qk_norm else None)
    model = gpu_model(P, cfg, glob, layers)
    ids = gen.token_ids(128, cfg.vocab, seed=4).numpy()
    bt = gen.block_table(8, 64, 8, 4, 2)
    pool = empty_pool(cfg, 64, fill_bits=0x7FA5)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    chunked(model, cfg, ids, [(0, 37), (37, 38), (38, 80), (80, 113), (113, 128)], bt, pool, err)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    check(cfg, glob, layers, ids, pool, bt)
    raw = pool.view(torch.int16).cpu().numpy()
    used = set(int(p) for p in bt[:8])
    assert all(np.all(raw[:, :, pg] == 0x7FA5) for pg in range(64) if pg not in used)


def test_mid_layer_shape_256_token_chunks(P):
    cfg = configs.MID.replace(n_layers=2, vocab=4096, name="mid-L2")
    glob, layers = gen.model_weights(cfg, seed=5, gain_sigma=0.1)
    model = gpu_model(P, cfg, glob, layers)
    n = 600
    ids = gen.token_ids(n, cfg.vocab, seed=5).numpy()
    bt = gen.block_table(38, 48, 38, 5, 2)
    pool = empty_pool(cfg, 48, fill_bits=0x7FA5)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    chunked(model, cfg, ids, [(0, 256), (256, 512), (512, n)], bt, pool, err)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    check(cfg, glob, layers, ids, pool, bt)


def test_short_chunks_over_long_prefix(P):
    """Chunks of at most 256 rows after a long first chunk: their query
    blocks are too few to fill the chip, so attention splits each block's
    keys over several workgroups (blocks with fewer key tiles than the
    longest leave their last splits empty) and merges the splits."""
    cfg = configs.MID.replace(n_layers=2, vocab=4096, name="mid-L2")
    glob, layers = gen.model_weights(cfg, seed=9, gain_sigma=0.1)
    model = gpu_model(P, cfg, glob, layers)
    n = 900
    ids = gen.token_ids(n, cfg.vocab, seed=9).numpy()
    bt = gen.block_table(57, 64, 57, 9, 2)
    pool = empty_pool(cfg, 64, fill_bits=0x7FA5)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    r1 = chunked(model, cfg, ids, [(0, 640), (640, 840), (840, 841), (841, 900)], bt, pool, err)
    whole = empty_pool(cfg, 64, fill_bits=0x7FA5)
    r1_whole = chunked(model, cfg, ids, [(0, n)], bt, whole, err)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    # Layer-local: layer 1 from the GPU's own input to it.  (Against the
    # end-to-end oracle, layer 1's K reaches about 1.1e-2 at this prefix,
    # for the undivided prefill too; the report line says how much of that
    # layer 0's rounding differences bring.)
    check_two_layers(cfg, glob, layers, ids, pool, bt, r1, n - 640, "chunked")
    check_two_layers(cfg, glob, layers, ids, whole, bt, r1_whole, n - 640, "undivided")
    # The split rows against the same rows of one undivided prefill.
    a, b = kv_logical(pool, bt, n)[:, :, 640:], kv_logical(whole, bt, n)[:, :, 640:]
    for l in range(cfg.n_layers):
        for kv in (0, 1):
            assert rel_err(a[l, kv], b[l, kv]) <= TOL


def test_large_layer_shape_short_chunks(P):
    """The large model's layer shape (8 query heads per KV head, head_dim
    128): calls with few query blocks split each GQA group over two 4-wave
    workgroups, and chunks of at most 256 rows also split the keys of each
    block over several workgroups.  A 300-row first chunk (split groups, no
    key splits), then 200-, 1- and 59-row chunks over it (split groups and
    key splits), against the oracle and against one undivided prefill."""
    cfg = configs.LARGE.replace(n_layers=2, vocab=4096, name="large-L2")
    glob, layers = gen.model_weights(cfg, seed=10, gain_sigma=0.1)
    model = gpu_model(P, cfg, glob, layers)
    n = 560
    ids = gen.token_ids(n, cfg.vocab, seed=10).numpy()
    bt = gen.block_table(35, 40, 35, 10, 2)
    pool = empty_pool(cfg, 40, fill_bits=0x7FA5)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    r1 = chunked(model, cfg, ids, [(0, 300), (300, 500), (500, 501), (501, n)], bt, pool, err)
    whole = empty_pool(cfg, 40, fill_bits=0x7FA5)
    r1_whole = chunked(model, cfg, ids, [(0, n)], bt, whole, err)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    check_two_layers(cfg, glob, layers, ids, pool, bt, r1, n - 300, "chunked")
    check_two_layers(cfg, glob, layers, ids, whole, bt, r1_whole, n - 300, "undivided")
    a, b = kv_logical(pool, bt, n)[:, :, 300:], kv_logical(whole, bt, n)[:, :, 300:]
    for l in range(cfg.n_layers):
        for kv in (0, 1):
            assert rel_err(a[l, kv], b[l, kv]) <= TOL


def test_several_sequences_at_different_starts(P):
    """One call prefills the second parts of three sequences whose first
    parts an earlier call wrote."""
    cfg = configs.MID.replace(n_layers=2, vocab=4096, name="mid-L2")
    glob, layers = gen.model_weights(cfg, seed=6, gain_sigma=0.1)
    model = gpu_model(P, cfg, glob, layers)
    lens, cuts = [150, 97, 260], [64, 5, 100]
    ids = [gen.token_ids(n, cfg.vocab, seed=6, stream=i).numpy() for i, n in enumerate(lens)]
    pages = [(n + 15) // 16 for n in lens]
    tables = gen.disjoint_block_tables(pages, 48, 17, 6, 3)
    d_bt = torch.tensor(tables, dtype=torch.int32, device=DEV)
    pool = empty_pool(cfg, 48, fill_bits=0x7FA5)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    ws = model.workspace(sum(lens), 3)
    for part in (0, 1):
        segs = [(0, c) if part == 0 else (c, n) for n, c in zip(lens, cuts)]
        cu = np.cumsum([0] + [b - a for a, b in segs]).tolist()
        flat = np.concatenate([x[a:b] for x, (a, b) in zip(ids, segs)])
        model.prefill_chunk(torch.tensor(flat, dtype=torch.int32, device=DEV), cu,
                            [a for a, _ in segs], d_bt, pool, ws, err)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    for x, bt in zip(ids, tables):
        check(cfg, glob, layers, x, pool, bt)


def test_aligned_chunks_equal_whole_prefill_bitwise(P):
    """Chunks of more than 256 rows starting at multiples of 32: every row
    runs the same GEMM and attention arithmetic as in one prefill over the
    whole prefix, so the cache bytes are equal."""
    cfg = configs.MID.replace(n_layers=3, vocab=4096, name="mid-L3")
    glob, layers = gen.model_weights(cfg, seed=7)
    model = gpu_model(P, cfg, glob, layers)
    n = 700
    ids = gen.token_ids(n, cfg.vocab, seed=7).numpy()
    bt = gen.block_table(44, 48, 44, 7, 1)
    d_bt = torch.tensor(np.asarray(bt)[None], dtype=torch.int32, device=DEV)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    whole = empty_pool(cfg, 48, fill_bits=0)
    model.prefill_prefix(torch.tensor(ids, dtype=torch.int32, device=DEV), [0, n], d_bt, whole,
                         model.workspace(n), err)
    parts = empty_pool(cfg, 48, fill_bits=0)
    chunked(model, cfg, ids, [(0, 288), (288, n)], bt, parts, err)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    np.testing.assert_array_equal(kv_logical(whole, bt, n), kv_logical(parts, bt, n))


def test_chunk_rejections(P):
    cfg = configs.TINY
    glob, layers = gen.model_weights(cfg, seed=8)
    model = gpu_model(P, cfg, glob, layers)
    pool = empty_pool(cfg, 8, fill_bits=0x7FA5)
    d_bt = torch.arange(8, dtype=torch.int32, device=DEV)[None]
    ids = torch.zeros(16, dtype=torch.int32, device=DEV)
    ws = model.workspace(16)
    with pytest.raises(P.PallasError) as e:
        model.prefill_chunk(ids, [0, 16], [120], d_bt, pool, ws)       # [120, 136) > 8 pages
    assert e.value.status == P.Status.OUT_OF_RANGE
    with pytest.raises(P.PallasError) as e:
        model.prefill_chunk(ids, [0, 16], [-1], d_bt, pool, ws)
    assert e.value.status == P.Status.INVALID_ARG
    torch.cuda.synchronize()
    assert torch.all(pool.view(torch.int16) == 0x7FA5)
