"""GPU parity of prefix prefill (K/V written into paged blocks) against the
oracle, element by element, within max|gpu - ref| <= 1e-2 max|ref| per
(layer, K|V) over the written positions; untouched slots keep their bytes.

Shapes: the 2-layer tiny decoder (full depth; QK-norm off and on); the mid
and large decoders' layer shapes at reduced depth and a 300-token prefix
(several 256-row GEMM tiles, a ragged tail, ten 32-query attention blocks);
several sequences of different lengths in one call; the causality property
(prefix K/V bitwise equal to the first rows of a longer prefill); one
sequence at the 32768-position limit (all of layer 0 and sampled rows of
layer 1 against the oracle)."""
import numpy as np
import pytest
import torch

from helpers import (TOL, empty_pool, ensure_lib, gpu_model, kv_logical, oracle_weights,
                     rel_err, shape_of)
from oracle import model as om
from workloads import configs, gen

pytestmark = pytest.mark.gpu
DEV = "cuda"


@pytest.fixture(scope="module")
def P():
    return ensure_lib()


def run_prefill(P, model, cfg, ids_list, tables, pages, fill=0x7FA5):
    pool = empty_pool(cfg, pages, fill_bits=fill)
    cu = [0]
    for ids in ids_list:
        cu.append(cu[-1] + len(ids))
    ids = torch.tensor(np.concatenate(ids_list), dtype=torch.int32, device=DEV)
    bt = torch.tensor(np.stack(tables), dtype=torch.int32, device=DEV)
    ws = model.workspace(cu[-1], len(ids_list))
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    model.prefill_prefix(ids, cu, bt, pool, ws, err)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    return pool


def check_against_oracle(cfg, glob, layers, ids, pool, bt, layers_to_check=None):
    g, ls = oracle_weights(glob, layers)
    shp = shape_of(cfg)
    L = cfg.n_layers if layers_to_check is None else layers_to_check
    K, V, _ = om.prefill(list(ids), g, ls, shp, n_layers=L)
    lv = kv_logical(pool, bt, len(ids))
    worst = 0.0
    for l in range(L):
        for kv, ref in ((0, K[l]), (1, V[l])):
            e = rel_err(lv[l, kv], ref)
            worst = max(worst, e)
            assert e <= TOL, f"layer {l} {'KV'[kv]}: rel err {e:.3g}"
    return worst


@pytest.mark.parametrize("qk_norm", [False, True])
def test_tiny_full_depth(P, qk_norm):
    cfg = configs.TINY.replace(qk_norm=qk_norm)
    glob, layers = gen.model_weights(cfg, seed=0, gain_sigma=0.1 if qk_norm else None)
    model = gpu_model(P, cfg, glob, layers)
    ids = gen.token_ids(128, cfg.vocab, seed=0).numpy()[:96]
    bt = gen.block_table(6, 64, 8, 0, 2)
    pool = run_prefill(P, model, cfg, [ids], [bt], 64)
    check_against_oracle(cfg, glob, layers, ids, pool, bt)
    # nothing outside the 96 written slots changed
    raw = pool.view(torch.int16).cpu().numpy()
    used = set(int(p) for p in bt[:6])
    for pg in range(64):
        if pg not in used:
            assert np.all(raw[:, :, pg] == 0x7FA5)


@pytest.mark.parametrize("p", [1, 15, 16, 17])
def test_tiny_page_boundary_lengths(P, p):
    """Prefixes of one token, and just below, at and just past one page."""
    cfg = configs.TINY.replace(qk_norm=True)
    glob, layers = gen.model_weights(cfg, seed=12, gain_sigma=0.1)
    model = gpu_model(P, cfg, glob, layers)
    ids = gen.token_ids(p, cfg.vocab, seed=12, stream=p).numpy()
    bt = gen.block_table(2, 8, 2, 12, p)
    pool = run_prefill(P, model, cfg, [ids], [bt], 8)
    check_against_oracle(cfg, glob, layers, ids, pool, bt)
    # slots past the prefix on its pages keep their bytes
    raw = pool.view(torch.int16).cpu().numpy()
    for t in range(p, 32):
        assert np.all(raw[:, :, bt[t // 16], t % 16] == 0x7FA5)


@pytest.mark.parametrize("shape", ["mid", "large"])
def test_layer_shapes_reduced_depth(P, shape):
    base = configs.preset(shape)
    cfg = base.replace(n_layers=2, vocab=4096, name=f"{shape}-L2")
    glob, layers = gen.model_weights(cfg, seed=1, gain_sigma=0.1)
    model = gpu_model(P, cfg, glob, layers)
    p = 300
    ids = gen.token_ids(p, cfg.vocab, seed=1).numpy()
    bt = gen.block_table(19, 40, 19, 1, 2)
    pool = run_prefill(P, model, cfg, [ids], [bt], 40)
    check_against_oracle(cfg, glob, layers, ids, pool, bt)


# The large model's attention shape (64 query heads over 8 KV heads,
# head_dim 128, QK-norm) with a narrower residual stream and FFN, so the
# oracle stays cheap; the projections still split K at 256 rows and below.
LARGE_HEADS = configs.LARGE.replace(n_layers=2, vocab=4096, hidden=1024, ffn=4096, name="large-heads-L2")


@pytest.mark.parametrize("p", [31, 32, 33, 64, 65, 256, 257])
def test_large_heads_boundary_lengths(P, p):
    """Prefixes around a 32-query block, a 64-key tile and the 256-row limit
    of the split-K projections and attention key splits (256 splits, 257
    does not)."""
    cfg = LARGE_HEADS
    glob, layers = gen.model_weights(cfg, seed=13, gain_sigma=0.1)
    model = gpu_model(P, cfg, glob, layers)
    ids = gen.token_ids(p, cfg.vocab, seed=13, stream=p).numpy()
    pages = (p + 15) // 16
    bt = gen.block_table(pages, pages + 4, pages, 13, p)
    pool = run_prefill(P, model, cfg, [ids], [bt], pages + 4)
    check_against_oracle(cfg, glob, layers, ids, pool, bt)


def test_large_heads_varlen_batch(P):
    """Five sequences in one call with 66 query blocks x 8 KV heads (528
    pairs): the undivided 8-head workgroups and the longest-first order
    across sequences, sequences of one token and of block and tile edges."""
    cfg = LARGE_HEADS
    glob, layers = gen.model_weights(cfg, seed=14, gain_sigma=0.1)
    model = gpu_model(P, cfg, glob, layers)
    lens = [1200, 1, 700, 65, 33]
    assert sum((n + 31) // 32 for n in lens) * cfg.n_kv_heads >= 512
    ids_list = [gen.token_ids(n, cfg.vocab, seed=14, stream=i).numpy() for i, n in enumerate(lens)]
    pages = [(n + 15) // 16 for n in lens]
    tables = gen.disjoint_block_tables(pages, 140, 80, 14, 5)
    pool = run_prefill(P, model, cfg, ids_list, list(tables), 140)
    for ids, bt in zip(ids_list, tables):
        check_against_oracle(cfg, glob, layers, ids, pool, bt)


def test_varlen_batch(P):
    cfg = configs.MID.replace(n_layers=2, vocab=4096, name="mid-L2")
    glob, layers = gen.model_weights(cfg, seed=2, gain_sigma=0.1)
    model = gpu_model(P, cfg, glob, layers)
    lens = [77, 1, 200, 33]
    ids_list = [gen.token_ids(n, cfg.vocab, seed=2, stream=i).numpy() for i, n in enumerate(lens)]
    pages = [(n + 15) // 16 for n in lens]
    tables = gen.disjoint_block_tables(pages, 40, 16, 2, 5)
    pool = run_prefill(P, model, cfg, ids_list, list(tables), 40)
    for ids, bt in zip(ids_list, tables):
        check_against_oracle(cfg, glob, layers, ids, pool, bt)


def test_causality_and_determinism(P):
    """K/V of a prefill over [0, p) equal, bit for bit, the first p positions
    of a prefill over [0, n); two identical calls give identical bytes."""
    cfg = configs.MID.replace(n_layers=3, vocab=4096, name="mid-L3")
    glob, layers = gen.model_weights(cfg, seed=3)
    model = gpu_model(P, cfg, glob, layers)
    n, p = 530, 403
    ids = gen.token_ids(n, cfg.vocab, seed=3).numpy()
    bt = gen.block_table(34, 40, 34, 3, 1)
    full = run_prefill(P, model, cfg, [ids], [bt], 40)
    pre = run_prefill(P, model, cfg, [ids[:p]], [bt], 40)
    pre2 = run_prefill(P, model, cfg, [ids[:p]], [bt], 40)
    a = kv_logical(full, bt, p)
    b = kv_logical(pre, bt, p)
    np.testing.assert_array_equal(a, b)
    assert torch.equal(pre.view(torch.int16), pre2.view(torch.int16))


def test_prefill_at_the_length_limit(P):
    """One sequence of PALLAS_MAX_PREFILL_LEN (32768) positions, the tiny
    decoder with QK-norm.  Layer 0's K/V depend on each token alone, so the
    oracle gives all 32768 rows; layer 1's K/V at sampled positions t (the
    first, page edges, the middle, the last) need one layer-0 attention row
    over the oracle's own layer-0 K/V of [0, t].  The first 300 rows also
    equal, bit for bit, those of a 300-token prefill."""
    cfg = configs.TINY.replace(qk_norm=True)
    glob, layers = gen.model_weights(cfg, seed=12, gain_sigma=0.1)
    model = gpu_model(P, cfg, glob, layers)
    n = 32768
    pages = n // 16
    ids = gen.token_ids(n, cfg.vocab, seed=12).numpy()
    bt = gen.block_table(pages, pages + 8, pages, 12, 1)
    pool = run_prefill(P, model, cfg, [ids], [bt], pages + 8)
    short = run_prefill(P, model, cfg, [ids[:300]], [bt], pages + 8)
    lv = kv_logical(pool, bt, n)
    np.testing.assert_array_equal(lv[:, :, :300], kv_logical(short, bt, 300))

    g, ls = oracle_weights(glob, layers)
    shp = shape_of(cfg)
    r = om.embed(list(ids), g)
    pos = np.arange(n)
    _, k0, v0 = om.layer(r, pos, None, None, ls[0], shp, om.bf16_round, kv_only=True)
    assert rel_err(lv[0, 0], k0) <= TOL
    assert rel_err(lv[0, 1], v0) <= TOL
    ts = [0, 1, 15, 16, 4095, 16384, 32735, 32767]
    k1, v1 = [], []
    for t in ts:
        r1, _, _ = om.layer(r[t:t + 1], pos[t:t + 1], k0[:t] if t else None, v0[:t] if t else None,
                            ls[0], shp, om.bf16_round)
        _, k, v = om.layer(r1, pos[t:t + 1], None, None, ls[1], shp, om.bf16_round, kv_only=True)
        k1.append(k[0])
        v1.append(v[0])
    assert rel_err(lv[1, 0, ts], np.stack(k1)) <= TOL
    assert rel_err(lv[1, 1, ts], np.stack(v1)) <= TOL


def test_profile_clock_samples_gemm_launches(P):
    """With timing on for the gate|up GEMM, a prefill records every one of
    its workgroups and a shader clock between 0.3 and 3.5 GHz; with timing
    off nothing is sampled."""
    cfg = configs.TINY
    glob, layers = gen.model_weights(cfg, seed=6)
    model = gpu_model(P, cfg, glob, layers)
    ids = gen.token_ids(300, cfg.vocab, seed=6).numpy()
    bt = gen.block_table(19, 24, 19, 6, 1)
    P.pallas_profile_reset()
    run_prefill(P, model, cfg, [ids], [bt], 24)
    assert P.pallas_profile_clock("gemm_gate_up") == (0.0, 0)
    P.pallas_profile_enable(["gemm_gate_up"])
    try:
        run_prefill(P, model, cfg, [ids], [bt], 24)
        ghz, wgs = P.pallas_profile_clock("gemm_gate_up")
    finally:
        P.pallas_profile_enable([])
        P.pallas_profile_reset()
    # 2 M tiles x 6 gate|up column groups of 128 would fill 12 of 256 CUs,
    # so the launch runs the smallest tiles: 2 x 192 rows x 11 groups of 64
    # columns.
    tiles = -(-300 // 192) * -(-cfg.ffn // 64)
    assert wgs == tiles * (cfg.n_layers - 1)
    assert 0.3 < ghz < 3.5
