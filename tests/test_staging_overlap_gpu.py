"""The transfer boundary and concurrent preparation on one GPU.

Wire staging (Section 5: suffix blocks leave the source GPU, cross the
network and are buffered at the target): chunks packed on the source side
go to pinned host memory, back to a target-side device arena, and are
assembled there; the assembled suffix equals the source's bit for bit.

Overlapped preparation (Section 4.3: prefix reconstruction and suffix
transfer proceed in parallel): the prefix prefill runs on one stream while
suffix chunks are assembled on another; the result equals the same work run
one call after the other, byte for byte.

Cancellation (Section 4.4: a change of the predicted target increments the
migration epoch and the obsolete attempt's blocks are discarded): after the
epoch moves on, chunks of the old epoch are rejected with nothing written,
and a fresh table assembled from the new epoch's chunks holds exactly the
source's suffix."""
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


class Req:
    """One request of the mid decoder's layer shape (2 layers): source full
    prefill of [0, n) into its own pool, suffix [p, n) packed in chunks."""

    def __init__(self, P, seed, n=300, p=200, chunk=32, pages=40):
        self.P = P
        self.cfg = cfg = configs.MID.replace(n_layers=2, vocab=4096, name="mid-L2")
        self.glob, self.layers = gen.model_weights(cfg, seed=seed, gain_sigma=0.1)
        self.model = gpu_model(P, cfg, self.glob, self.layers)
        self.n, self.p = n, p
        self.ids = gen.token_ids(n, cfg.vocab, seed=seed).numpy()
        need = (n + 15) // 16
        self.src_bt = gen.block_table(need, pages, need, seed, 1)
        self.dst_bt = gen.block_table(need, pages, need, seed, 2)
        self.d_src_bt = torch.tensor(self.src_bt, dtype=torch.int32, device=DEV)
        self.d_dst_bt = torch.tensor(self.dst_bt, dtype=torch.int32, device=DEV)
        self.pages = pages
        self.err = torch.zeros(1, dtype=torch.int32, device=DEV)
        self.src = empty_pool(cfg, pages, fill_bits=0)
        self.model.prefill_prefix(torch.tensor(self.ids, dtype=torch.int32, device=DEV), [0, n],
                                  self.d_src_bt[None], self.src, self.model.workspace(n), self.err)
        self.row = 2 * cfg.n_layers * cfg.n_kv_heads * cfg.head_dim * 2
        self.pieces = [(t, min(chunk, n - t), (t - p) * self.row) for t in range(p, n, chunk)]
        self.arena = torch.empty((n - p) * self.row, dtype=torch.uint8, device=DEV)
        P.pallas_pack_suffix_blocks(self.src, self.d_src_bt,
                                    [P.ChunkDesc(s, c, o) for s, c, o in self.pieces], self.arena, self.err)
        torch.cuda.synchronize()

    def headers(self, epoch, req=5):
        c = self.cfg
        return [self.P.ChunkHeader(req, epoch, s, k, o, c.n_layers, c.n_kv_heads, c.head_dim, 2)
                for s, k, o in self.pieces]


def test_pinned_host_staging_is_bit_exact(P):
    r = Req(P, seed=21)
    host = torch.empty(r.arena.numel(), dtype=torch.uint8, pin_memory=True)
    host.copy_(r.arena, non_blocking=True)            # device -> pinned host
    target_arena = torch.empty_like(r.arena)
    target_arena.copy_(host, non_blocking=True)       # pinned host -> device
    dst = empty_pool(r.cfg, r.pages, fill_bits=0x7FA5)
    P.pallas_assemble_kv(dst, r.d_dst_bt, r.headers(1), target_arena, 5, 1, r.err)
    torch.cuda.synchronize()
    assert int(r.err.item()) == 0
    np.testing.assert_array_equal(kv_logical(dst, r.dst_bt, r.n)[:, :, r.p:],
                                  kv_logical(r.src, r.src_bt, r.n)[:, :, r.p:])
    # pages the suffix does not touch keep the sentinel
    used = set(int(x) for x in r.dst_bt[r.p // 16:])
    raw = dst.view(torch.int16).cpu().numpy()
    assert all(np.all(raw[:, :, pg] == 0x7FA5) for pg in range(r.pages) if pg not in used)


def test_prefill_and_assembly_on_two_streams(P):
    """Prefix prefill on stream A while 32-token chunks are assembled one
    launch each on stream B; compared with the sequential order."""
    r = Req(P, seed=22)
    a, b = torch.cuda.Stream(), torch.cuda.Stream()
    ids = torch.tensor(r.ids[:r.p], dtype=torch.int32, device=DEV)
    ws = r.model.workspace(r.p)
    hdrs = r.headers(3)

    def run(concurrent):
        dst = empty_pool(r.cfg, r.pages, fill_bits=0x7FA5)
        err = torch.zeros(1, dtype=torch.int32, device=DEV)
        torch.cuda.synchronize()
        sa = a if concurrent else torch.cuda.current_stream()
        sb = b if concurrent else torch.cuda.current_stream()
        with torch.cuda.stream(sa):
            r.model.prefill_prefix(ids, [0, r.p], r.d_dst_bt[None], dst, ws, err, stream=sa)
        for h in hdrs:
            P.pallas_assemble_kv(dst, r.d_dst_bt, [h], r.arena, 5, 3, err, stream=sb)
        torch.cuda.synchronize()
        assert int(err.item()) == 0
        return dst

    seq, conc = run(False), run(True)
    assert torch.equal(seq.view(torch.int16), conc.view(torch.int16))
    lv = kv_logical(conc, r.dst_bt, r.n)
    np.testing.assert_array_equal(lv[:, :, r.p:], kv_logical(r.src, r.src_bt, r.n)[:, :, r.p:])
    g, ls = oracle_weights(r.glob, r.layers)
    K, V, _ = om.prefill(list(r.ids[:r.p]), g, ls, shape_of(r.cfg))
    for l in range(r.cfg.n_layers):
        assert rel_err(lv[l, 0, :r.p], K[l]) <= TOL and rel_err(lv[l, 1, :r.p], V[l]) <= TOL


def test_epoch_cancellation_mid_stream(P):
    r = Req(P, seed=23)
    dst = empty_pool(r.cfg, r.pages, fill_bits=0x7FA5)
    old = r.headers(epoch=1)
    half = len(old) // 2
    # epoch 1: the first half of the chunks arrives and is assembled
    P.pallas_assemble_kv(dst, r.d_dst_bt, old[:half], r.arena, 5, 1, r.err)
    torch.cuda.synchronize()
    # the predicted target changes: epoch 2; the old attempt's table is
    # released and a new one allocated
    new_bt = gen.block_table((r.n + 15) // 16, r.pages, (r.n + 15) // 16, 23, 9)
    d_new_bt = torch.tensor(new_bt, dtype=torch.int32, device=DEV)
    before = dst.clone()
    # late epoch-1 chunks are rejected and write nothing
    with pytest.raises(P.PallasError) as e:
        P.pallas_assemble_kv(dst, d_new_bt, old[half:], r.arena, 5, 2, r.err)
    assert e.value.status == P.Status.STALE_EPOCH
    # a batch mixing epochs is rejected as a whole
    with pytest.raises(P.PallasError):
        P.pallas_assemble_kv(dst, d_new_bt, r.headers(2)[:1] + old[half:half + 1], r.arena, 5, 2, r.err)
    torch.cuda.synchronize()
    assert torch.equal(before.view(torch.int16), dst.view(torch.int16))
    # the new epoch's chunks go into the new table
    fresh = empty_pool(r.cfg, r.pages, fill_bits=0x7FA5)
    hdrs = r.headers(epoch=2)
    P.pallas_assemble_kv(fresh, d_new_bt, hdrs, r.arena, 5, 2, r.err)
    torch.cuda.synchronize()
    assert int(r.err.item()) == 0
    assert P.pallas_check_coverage(r.p, [h.start_pos for h in hdrs], [h.num_tokens for h in hdrs],
                                   r.n) == P.Status.OK
    np.testing.assert_array_equal(kv_logical(fresh, new_bt, r.n)[:, :, r.p:],
                                  kv_logical(r.src, r.src_bt, r.n)[:, :, r.p:])
    # only the suffix's pages of the new table were written
    used = set(int(x) for x in new_bt[r.p // 16:])
    raw = fresh.view(torch.int16).cpu().numpy()
    assert all(np.all(raw[:, :, pg] == 0x7FA5) for pg in range(r.pages) if pg not in used)
