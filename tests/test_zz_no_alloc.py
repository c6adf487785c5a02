"""pallas_decode_step_static (the decode step without a workspace, over the
library's per-GPU static scratch) against pallas_decode_step on the same
inputs, called through the C ABI: two calls in a row, the second with fewer
sequences at smaller positions, so it runs over the scratch the first one
left.  Logits and the K/V each step writes must equal the workspace entry
point's bit for bit (the same kernels with the same split counts), which is
within the 1e-2 max|ref| bar.

The model has the large decoder's layer shape (2 layers, hidden 5120, 64/8
heads, ffn 25600) and the full 151936-token vocabulary, so the skinny O and
down projections split K over workgroups and count arrivals in the
scratch's counters, and attention runs up to 33 key splits."""
import numpy as np
import pytest
import torch

from helpers import TOL, empty_pool, ensure_lib, gpu_model, rel_err
from workloads import configs, gen

pytestmark = pytest.mark.gpu
DEV = "cuda"


@pytest.fixture(scope="module")
def P():
    return ensure_lib()


def test_static_scratch_decode_matches_workspace_decode(P):
    cfg = configs.LARGE.replace(n_layers=2, name="large-L2")
    glob, layers = gen.model_weights(cfg, seed=51, gain_sigma=0.1, device=DEV)
    model = gpu_model(P, cfg, glob, layers)
    lens = [700, 2100, 33, 1500, 0, 300, 41]
    calls = [[0, 1, 2, 3, 4], [5, 6]]   # sequences decoded by the first and the second call
    ids = [gen.token_ids(n + 1, cfg.vocab, seed=51, stream=i).numpy() for i, n in enumerate(lens)]
    pages = [(n + 1 + 15) // 16 for n in lens]
    tables = gen.disjoint_block_tables(pages, sum(pages), max(pages), 51, 1)
    d_bt = torch.tensor(tables, dtype=torch.int32, device=DEV)
    pool = empty_pool(cfg, sum(pages), fill_bits=0)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    pre = [i for i, n in enumerate(lens) if n > 0]
    cu = np.cumsum([0] + [lens[i] for i in pre]).tolist()
    flat = torch.tensor(np.concatenate([ids[i][:lens[i]] for i in pre]), dtype=torch.int32, device=DEV)
    ws = model.workspace(cu[-1], len(pre))
    model.prefill_prefix(flat, cu, d_bt[pre], pool, ws, err)
    torch.cuda.synchronize()
    snapshot = pool.clone()

    def args(seqs):
        toks = torch.tensor([ids[i][lens[i]] for i in seqs], dtype=torch.int32, device=DEV)
        return toks, [lens[i] for i in seqs], d_bt[seqs].contiguous()

    # Reference: the workspace entry point, the same two calls.
    wsd = model.workspace(len(calls[0]), len(calls[0]))
    ref = []
    for seqs in calls:
        toks, pos, bt = args(seqs)
        out = torch.empty((len(seqs), cfg.vocab), dtype=torch.float32, device=DEV)
        model.decode_step(toks, pos, bt, pool, out, wsd, err)
        ref.append(out)
    torch.cuda.synchronize()
    pool_ref = pool.clone()
    # The static-scratch entry point: the two calls back to back.
    pool.copy_(snapshot)
    got = []
    for seqs in calls:
        toks, pos, bt = args(seqs)
        out = torch.full((len(seqs), cfg.vocab), float("nan"), dtype=torch.float32, device=DEV)
        model.decode_step_static(toks, pos, bt, pool, out, err)
        got.append(out)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    for c, (a, b) in enumerate(zip(got, ref)):
        for i in range(a.shape[0]):
            assert rel_err(a[i].double().cpu().numpy(), b[i].double().cpu().numpy()) <= TOL, f"call {c} row {i}"
        assert torch.equal(a, b), f"call {c}: logits differ from the workspace entry point"
    assert torch.equal(pool, pool_ref), "the K/V written differ from the workspace entry point"
