#!/usr/bin/env python3
"""Benchmark of target-side KV-cache reconstruction on one MI355X.

One step is one pass of the whole reconstruction path over the workload:

  1. prefix prefill of every request's prefix [0, p_i) into the target pool
     (K/V written into 16-token pages through the target block tables);
  2. pack of every request's suffix [p_i, n_i) out of the source pool into
     contiguous per-layer transfer chunks;
  3. assembly of those chunks into the target block tables;
  4. one batched decode step at positions n_i over the assembled caches.

Inputs are synthetic and resident in device memory before timing starts:
random-init bf16 weights N(0, 0.02) of the workload's decoder shape, uniform
token ids, shuffled block tables; the source pool holds the K/V of a
source-side full prefill of [0, n_i) (run once, untimed).

The printed JSON line reports prefix tokens per second over the whole step,
the per-phase breakdown (prefill tokens/s and fraction of the bf16 MFMA
peak, pack/assemble GB/s and fraction of the HBM peak), the roofline of the
dominant kernel (the gate|up projection GEMM, timed with HIP events on the
launch stream inside the timed region), and the CPU oracle timed on a
bounded sample on this host.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBPS = 8000.0      # MI355X HBM3E
NOMINAL_SCLK_GHZ = 2.4      # clock the MFMA peak is quoted at

# Memory-side traffic of one gate|up GEMM launch at the large workload, from
# two rocprofv3 --pmc passes over `bench.py --steps 1 --warmup 0
# --no-cpu-baseline --no-stress --no-chunked --no-staging` (FETCH_SIZE, then
# WRITE_SIZE, KiB per dispatch, averaged over the gate|up launches at
# M = 3000; profiles/gemm_attention_counters.md), each scaled by what the same counter
# reads for a 1 GiB device copy (`bench.py --copy-calibration`: FETCH_SIZE
# x 2.0, WRITE_SIZE x 1.0).  Valid
# only for the GEMM source it was measured on: a different csrc/gemm.hip
# reports null.
GEMM_TRAFFIC = {
    "gemm_source_sha256_16": "02fe53aa9dc84ac5",
    "fetch_kib": 1.34892e6, "fetch_scale": 2.0,
    "write_kib": 1.94010e5, "write_scale": 1.0,
}


def gemm_traffic_bytes():
    import hashlib
    src = os.path.join(ROOT, "paper_2608_16477_amd", "csrc", "gemm.hip")
    sha = hashlib.sha256(open(src, "rb").read()).hexdigest()[:16]
    t = GEMM_TRAFFIC
    if sha != t["gemm_source_sha256_16"]:
        return None
    return (t["fetch_kib"] * t["fetch_scale"] + t["write_kib"] * t["write_scale"]) * 1024.0

# Memory-side traffic of pack and assemble (kv_copy_kernel) for the large
# workload's 1000-token suffix, from the same two counter passes and the
# same calibration (profiles/kv_copy_traffic.md), KiB per launch after
# scaling: FETCH_SIZE x 2.0, WRITE_SIZE x 1.0.  Valid only for the copy
# source it was measured on.
COPY_TRAFFIC = {
    "copy_source_sha256_16": "09274b976938982d",
    "tokens": 1000,
    "pack": {"fetch_kib": 256139.0, "write_kib": 256000.0},
    "assemble": {"fetch_kib": 256143.0, "write_kib": 256000.0},
}


def copy_traffic_bytes(kind, suffix_tokens):
    """HBM bytes of one pack or assemble launch from the stored counters, or
    None for another copy source or suffix length."""
    import hashlib
    src = os.path.join(ROOT, "paper_2608_16477_amd", "csrc", "kv_copy.hip")
    sha = hashlib.sha256(open(src, "rb").read()).hexdigest()[:16]
    t = COPY_TRAFFIC
    if sha != t["copy_source_sha256_16"] or suffix_tokens != t["tokens"]:
        return None
    return (t[kind]["fetch_kib"] + t[kind]["write_kib"]) * 1024.0


METRIC = "prefix-prefill tokens/s + % bf16 MFMA peak; KV pack/assemble GB/s + % HBM peak"


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="large",
                    choices=["tiny", "mid", "large", "large-aligned", "concurrent"])
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-stress", action="store_true",
                    help="skip the stress-layout copy measurements (suffixes of 64-4096 tokens)")
    ap.add_argument("--no-chunked", action="store_true",
                    help="skip the chunked-prefill measurements (256-token chunks, with 0-3 "
                         "resident decode sessions interleaved) and the post-handover recompute legs")
    ap.add_argument("--no-staging", action="store_true",
                    help="skip the pinned-host staging legs and the two-stream overlap measurements "
                         "(back to back and paced at 100-500 Mbps)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="run one 1 GiB device-to-device copy and exit (the reference "
                         "point for scaling FETCH_SIZE / WRITE_SIZE counter readings)")
    return ap.parse_args()


def copy_calibration():
    """One plain copy of known size: 2^28 int32 (1 GiB read, 1 GiB written)."""
    import torch
    n = (1 << 30) // 4
    a = torch.ones(n, dtype=torch.int32, device="cuda")
    b = torch.empty_like(a)
    torch.cuda.synchronize()
    b.copy_(a)
    torch.cuda.synchronize()
    print(f"[bench] copied {n * 4} bytes", file=sys.stderr, flush=True)


def load_library():
    import paper_2608_16477_amd as P
    if not os.path.exists(P.library_path()):
        from paper_2608_16477_amd import build
        build.build()
    P.lib()
    return P


class Setup:
    """Device-resident inputs of one workload."""

    def __init__(self, P, wl, seed):
        import numpy as np
        import torch
        from workloads import gen

        self.P, self.wl, self.cfg = P, wl, wl.model
        cfg, dev = self.cfg, "cuda"
        self.glob, self.layers = gen.model_weights(cfg, seed=seed, device=dev)
        self.model = P.Model(cfg, self.glob, self.layers)
        B = wl.num_seqs
        self.ns, self.ps = list(wl.ctx), list(wl.prefix)
        self.ids = [gen.token_ids(n + 1, cfg.vocab, seed=seed, stream=i).numpy()
                    for i, n in enumerate(self.ns)]
        src_pages = [wl.pages_for(n) for n in self.ns]
        dst_pages = [wl.pages_for(n + 1) for n in self.ns]
        self.max_pages = max(dst_pages)
        src_pool_pages, dst_pool_pages = sum(src_pages), sum(dst_pages)
        self.src_tab = torch.tensor(gen.disjoint_block_tables(src_pages, src_pool_pages, self.max_pages,
                                                              seed, 1), dtype=torch.int32, device=dev)
        self.dst_tab = torch.tensor(gen.disjoint_block_tables(dst_pages, dst_pool_pages, self.max_pages,
                                                              seed, 2), dtype=torch.int32, device=dev)
        shape = (cfg.n_layers, 2, 0, cfg.page_size, cfg.n_kv_heads, cfg.head_dim)
        self.src = torch.zeros(shape[:2] + (src_pool_pages,) + shape[3:], dtype=torch.bfloat16, device=dev)
        self.dst = torch.zeros(shape[:2] + (dst_pool_pages,) + shape[3:], dtype=torch.bfloat16, device=dev)
        self.err = torch.zeros(1, dtype=torch.int32, device=dev)
        self.prefix_ids = torch.tensor(np.concatenate([ids[:p] for ids, p in zip(self.ids, self.ps)]),
                                       dtype=torch.int32, device=dev)
        self.cu = [0]
        for p in self.ps:
            self.cu.append(self.cu[-1] + p)
        self.tokens = torch.tensor([ids[n] for ids, n in zip(self.ids, self.ns)], dtype=torch.int32,
                                   device=dev)
        self.logits = torch.empty((B, cfg.vocab), dtype=torch.float32, device=dev)
        self.ws = self.model.workspace(max(self.cu[-1], max(self.ns)), B)
        # suffix chunks per request
        row = 2 * cfg.n_layers * cfg.n_kv_heads * cfg.head_dim * 2
        self.row_bytes = row
        self.descs, self.hdrs = [], []
        off = 0
        for i, (n, p) in enumerate(zip(self.ns, self.ps)):
            step = wl.chunk_tokens or (n - p)
            d, h = [], []
            for t in range(p, n, step):
                c = min(step, n - t)
                d.append(P.ChunkDesc(t, c, off))
                h.append(P.ChunkHeader(1000 + i, 1, t, c, off, cfg.n_layers, cfg.n_kv_heads,
                                       cfg.head_dim, 2))
                off += c * row
            self.descs.append(d)
            self.hdrs.append(h)
        self.arena = torch.empty(max(off, 16), dtype=torch.uint8, device=dev)
        self.suffix_tokens = sum(n - p for n, p in zip(self.ns, self.ps))
        # source cache: full prefill of [0, n_i), untimed
        for i, n in enumerate(self.ns):
            self.model.prefill_prefix(torch.tensor(self.ids[i][:n], dtype=torch.int32, device=dev), [0, n],
                                      self.src_tab[i:i + 1], self.src, self.ws, self.err)
        torch.cuda.synchronize()

    def prefill(self):
        self.model.prefill_prefix(self.prefix_ids, self.cu, self.dst_tab, self.dst, self.ws, self.err)

    def pack(self):
        for i in range(self.wl.num_seqs):
            self.P.pallas_pack_suffix_blocks(self.src, self.src_tab[i], self.descs[i], self.arena, self.err)

    def assemble(self):
        for i in range(self.wl.num_seqs):
            self.P.pallas_assemble_kv(self.dst, self.dst_tab[i], self.hdrs[i], self.arena, 1000 + i, 1,
                                      self.err)

    def decode(self):
        self.model.decode_step(self.tokens, self.ns, self.dst_tab, self.dst, self.logits, self.ws, self.err)


def copies_stress(P, seed):
    """Pack and assemble at the stress layout: an 8192-token source of
    N(0,1) K/V in 512 shuffled pages, a 1024-page target pool with half its
    pages occupied, suffixes of 64-4096 tokens moved as in-order 32-token
    chunks, all chunks of one suffix in one launch.  Ten warm-up calls, then
    the median of 50 event-timed calls per figure; one more row times one
    launch per 32-token chunk.  Each row also times a plain contiguous device
    copy of the same payload (torch's copy kernel): the practical ceiling.
    Up to about 256 MB read + written the MI355X's 256 MB last-level cache
    absorbs the writes; above it a plain copy runs at about 0.64 of peak."""
    import numpy as np
    import torch
    from workloads import configs, gen

    cfg = configs.STRESS_KV
    L, hkv, d = cfg.n_layers, cfg.n_kv_heads, cfg.head_dim
    n_src = configs.STRESS_SOURCE_TOKENS
    src_pages = n_src // cfg.page_size
    tp = configs.STRESS_TARGET_PAGES
    src = gen.kv_pool_normal(L, src_pages, cfg.page_size, hkv, d, seed=seed, device="cuda")
    src_bt = torch.from_numpy(gen.block_table(src_pages, src_pages, src_pages, seed, 1)).cuda()
    occupied = np.sort(gen.permutation(tp, seed, 2)[: tp // 2])
    free = np.setdiff1d(np.arange(tp), occupied).astype(np.int32)
    dst = torch.empty((L, 2, tp, cfg.page_size, hkv, d), dtype=torch.bfloat16, device="cuda")
    dst.view(torch.int16).fill_(gen.SENTINEL_BITS)
    dst_bt = torch.from_numpy(gen.block_table(src_pages, tp, src_pages, seed, 3, free_pages=free)).cuda()
    row = cfg.s_kv
    arena = torch.empty(max(configs.STRESS_SUFFIXES) * row, dtype=torch.uint8, device="cuda")
    err = torch.zeros(1, dtype=torch.int32, device="cuda")

    def median_us(fn, reps=50, warm=10):
        for _ in range(warm):
            fn()
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in range(reps)]
        for a, b in evs:
            a.record()
            fn()
            b.record()
        torch.cuda.synchronize()
        return float(np.median([a.elapsed_time(b) for a, b in evs])) * 1e3

    def same(a, b, what):
        if not torch.equal(a.view(torch.uint8), b.view(torch.uint8)):
            raise RuntimeError(f"graph replay of {what} differs from the eager call")

    def graph_us(fn, check, calls=20, reps=10):
        """Device time per call: `calls` calls captured in one graph (the
        copies enqueue no memset and allocate nothing), the graph replayed
        back to back; median over `reps` event-timed replays, divided by
        `calls`.  The host-side marshalling that the single-call figure
        includes is outside.  `check()` compares the replayed result with
        the eager one, before and after the timed replays."""
        fn()
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for _ in range(calls):
                fn()
        g.replay()
        torch.cuda.synchronize()
        check()
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in range(reps)]
        for a, b in evs:
            a.record()
            g.replay()
            b.record()
        torch.cuda.synchronize()
        check()
        del g
        return float(np.median([a.elapsed_time(b) for a, b in evs])) * 1e3 / calls

    rows = []
    for s in configs.STRESS_SUFFIXES:
        start = n_src - s
        descs, hdrs = [], []
        for k, t in enumerate(range(start, n_src, configs.STRESS_CHUNK)):
            c = min(configs.STRESS_CHUNK, n_src - t)
            descs.append(P.ChunkDesc(t, c, k * configs.STRESS_CHUNK * row))
            hdrs.append(P.ChunkHeader(7, 1, t, c, k * configs.STRESS_CHUNK * row, L, hkv, d, 2))
        nbytes = 2 * s * row
        do_pack = lambda: P.pallas_pack_suffix_blocks(src, src_bt, descs, arena, err)
        do_asm = lambda: P.pallas_assemble_kv(dst, dst_bt, hdrs, arena, 7, 1, err)
        t_pack = median_us(do_pack)
        t_asm = median_us(do_asm)
        # practical ceiling: a plain contiguous device copy of the same payload
        # (torch's copy kernel), timed the same way
        ca = arena[: s * row]
        cb = torch.empty_like(ca)
        t_copy = median_us(lambda: cb.copy_(ca))
        # the same three, replayed from a graph
        packed = ca.clone()
        dst_pages = dst_bt[start // cfg.page_size: n_src // cfg.page_size].long()
        assembled = dst[:, :, dst_pages].clone()

        g_pack = graph_us(do_pack, lambda: same(ca, packed, "pack"))
        g_asm = graph_us(do_asm, lambda: same(dst[:, :, dst_pages], assembled, "assemble"))
        g_copy = graph_us(lambda: cb.copy_(ca), lambda: same(cb, ca, "device copy"))
        del cb, packed, assembled
        frac = lambda us: nbytes / us / 1e3 / PEAK_HBM_GBPS
        rows.append({"suffix_tokens": s, "chunks_per_launch": len(descs), "bytes": nbytes,
                     "pack_us": t_pack, "pack_GBps": nbytes / t_pack / 1e3,
                     "pack_hbm_frac": frac(t_pack),
                     "assemble_us": t_asm, "assemble_GBps": nbytes / t_asm / 1e3,
                     "assemble_hbm_frac": frac(t_asm),
                     "device_copy_us": t_copy, "device_copy_hbm_frac": frac(t_copy),
                     "graph": {"pack_us": g_pack, "pack_hbm_frac": frac(g_pack),
                               "assemble_us": g_asm, "assemble_hbm_frac": frac(g_asm),
                               "device_copy_us": g_copy, "device_copy_hbm_frac": frac(g_copy)}})
    # one launch per 32-token chunk
    c = configs.STRESS_CHUNK
    one_d = [P.ChunkDesc(n_src - c, c, 0)]
    one_h = [P.ChunkHeader(7, 1, n_src - c, c, 0, L, hkv, d, 2)]
    one_pack = lambda: P.pallas_pack_suffix_blocks(src, src_bt, one_d, arena, err)
    one_asm = lambda: P.pallas_assemble_kv(dst, dst_bt, one_h, arena, 7, 1, err)
    lat = {"chunk_tokens": c, "bytes": 2 * c * row,
           "pack_us": median_us(one_pack), "assemble_us": median_us(one_asm)}
    packed = arena[: c * row].clone()
    pages = dst_bt[(n_src - c) // cfg.page_size: n_src // cfg.page_size].long()
    assembled = dst[:, :, pages].clone()
    lat["graph_pack_us"] = graph_us(one_pack, lambda: same(arena[: c * row], packed, "pack"))
    lat["graph_assemble_us"] = graph_us(one_asm, lambda: same(dst[:, :, pages], assembled, "assemble"))
    torch.cuda.synchronize()
    assert int(err.item()) == 0, "device-side error flag raised in the stress copies"
    return {"layout": (f"{L} layers, {hkv} KV heads, head_dim {d}: {n_src}-token source in "
                       f"{src_pages} shuffled pages; {tp}-page target, half occupied; "
                       f"{c}-token chunks"), "rows": rows, "per_chunk_launch": lat}


def chunked_prefill(st, chunk=256, residents=(0, 1, 2, 3), reps=3, resident_ctx=2000):
    """The workload's first prefix prefilled in `chunk`-token chunks
    (pallas_prefill_chunk), each chunk attending to the earlier chunks
    through the target pool; then the same with R resident sessions
    interleaved, one batched decode step of the R residents after every
    chunk (the concurrency experiment's contention with resident
    decoding).  The residents decode over their own `resident_ctx`-token
    caches in a separate pool (N(0,1) bf16 K/V).  Median of `reps` runs
    after one warm-up; the whole prefix's time, migration tokens/s, and the
    residents' mean decode-step time."""
    import numpy as np
    import torch
    from workloads import gen

    P, cfg, model = st.P, st.cfg, st.model
    p = st.ps[0]
    ids = torch.tensor(st.ids[0][:p], dtype=torch.int32, device="cuda")
    bt = st.dst_tab[:1]
    bounds = [(a, min(a + chunk, p)) for a in range(0, p, chunk)]
    ws = model.workspace(chunk, max(1, max(residents)))
    err = st.err
    rmax = max(residents)
    if rmax:
        rpages = (resident_ctx + 1 + 15) // 16
        rpool = gen.kv_pool_normal(cfg.n_layers, rmax * rpages, cfg.page_size, cfg.n_kv_heads,
                                   cfg.head_dim, seed=11, device="cuda")
        rtab = torch.arange(rmax * rpages, dtype=torch.int32, device="cuda").view(rmax, rpages)
        rtok = torch.randint(0, cfg.vocab, (rmax,), dtype=torch.int32, device="cuda")
        rlog = torch.empty((rmax, cfg.vocab), dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream()

    def run(R, evs=None):
        for k, (a, b) in enumerate(bounds):
            model.prefill_chunk(ids[a:b], [0, b - a], [a], bt, st.dst, ws, err)
            if R:
                if evs is not None:
                    evs[k][0].record(stream)
                model.decode_step(rtok[:R], [resident_ctx] * R, rtab[:R], rpool, rlog[:R], ws, err)
                if evs is not None:
                    evs[k][1].record(stream)

    flops = cfg.prefill_flops(p)
    out = {"chunk_tokens": chunk, "prefix_tokens": p, "chunks": len(bounds), "rows": []}
    for R in residents:
        run(R)
        times, itl = [], []
        for _ in range(reps):
            evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
                   for _ in bounds]
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            run(R, evs)
            b.record(stream)
            torch.cuda.synchronize()
            times.append(a.elapsed_time(b))
            if R:
                itl.append(float(np.mean([x.elapsed_time(y) for x, y in evs])))
        ms = float(np.median(times))
        row = {"residents": R, "ms": ms, "migration_tokens_per_s": p / ms * 1e3}
        if R == 0:
            row["tflops"] = flops / ms / 1e9
            row["mfma_frac"] = flops / ms / 1e9 / PEAK_BF16_TFLOPS
        else:
            row["resident_decode_step_ms"] = float(np.median(itl))
        out["rows"].append(row)
    # one more pass without residents, with events around every launch
    P.pallas_profile_reset()
    P.pallas_profile_enable(P.KERNEL_CLASSES)
    run(0)
    torch.cuda.synchronize()
    prof = P.pallas_profile_read()
    P.pallas_profile_enable([])
    P.pallas_profile_reset()
    out["kernels_ms"] = {k: v[0] for k, v in prof.items() if v[1]}
    torch.cuda.synchronize()
    assert int(err.item()) == 0, "device-side error flag raised in the chunked prefill"
    return out


def post_handover_recompute(st, assemble_ms, reps=3, chunk=256):
    """What the target pays after handover when a suffix is recomputed
    instead of migrated (the "w/o SM" variant of the ablation study, Sec.
    6.5), and when the whole history is (the recomputation baseline): the
    first request's suffix [p, n) prefilled over its prefix K/V already in
    the target pool (pallas_prefill_chunk, as one call and in `chunk`-token
    chunks), and a prefill of all n tokens.  Median of `reps` runs after
    one warm-up, against assembling the migrated suffix (`assemble_ms`)."""
    import numpy as np
    import torch

    model, stream = st.model, torch.cuda.current_stream()
    n, p = st.ns[0], st.ps[0]
    ids = torch.tensor(st.ids[0][:n], dtype=torch.int32, device="cuda")
    bt = st.dst_tab[:1]

    def suffix_one():
        model.prefill_chunk(ids[p:n], [0, n - p], [p], bt, st.dst, st.ws, st.err)

    def suffix_chunks():
        for a in range(p, n, chunk):
            b = min(a + chunk, n)
            model.prefill_chunk(ids[a:b], [0, b - a], [a], bt, st.dst, st.ws, st.err)

    def history():
        model.prefill_prefix(ids, [0, n], bt, st.dst, st.ws, st.err)

    def median_ms(fn):
        fn()
        times = []
        for _ in range(reps):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            fn()
            b.record(stream)
            torch.cuda.synchronize()
            times.append(a.elapsed_time(b))
        return float(np.median(times))

    out = {"prefix_tokens": p, "suffix_tokens": n - p, "assemble_ms": assemble_ms}
    for name, fn, tokens in (("suffix_one_call", suffix_one, n - p),
                             (f"suffix_chunks_{chunk}", suffix_chunks, n - p),
                             ("whole_history", history, n)):
        ms = median_ms(fn)
        out[name] = {"ms": ms, "tokens_per_s": tokens / ms * 1e3,
                     "vs_assemble": ms / assemble_ms if assemble_ms > 0 else None}
    torch.cuda.synchronize()
    assert int(st.err.item()) == 0, "device-side error flag raised in the recompute legs"
    return out


def wire_staging(st, reps=10):
    """The transfer boundary through host memory: the suffix packed on the
    source side, copied to pinned host memory, copied back to a target-side
    device arena and assembled -- once as one chunk holding the whole suffix
    and once for a single 32-token chunk.  Per leg: median time of `reps`
    runs (HIP events on the current stream) and its rate over the chunk's
    payload bytes (each leg moves the payload once); the PCIe-inclusive rate
    is the payload over the sum of the legs."""
    import numpy as np
    import torch

    P, cfg = st.P, st.cfg
    stream = torch.cuda.current_stream()
    n, p = st.ns[0], st.ps[0]
    out = {}
    for name, count in (("suffix", n - p), ("chunk32", 32)):
        nbytes = count * st.row_bytes
        src_arena = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
        dst_arena = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
        host = torch.empty(nbytes, dtype=torch.uint8, pin_memory=True)
        desc = [P.ChunkDesc(p, count, 0)]
        hdr = [P.ChunkHeader(1000, 1, p, count, 0, cfg.n_layers, cfg.n_kv_heads, cfg.head_dim, 2)]
        legs = {"pack": lambda: P.pallas_pack_suffix_blocks(st.src, st.src_tab[0], desc, src_arena, st.err),
                "d2h": lambda: host.copy_(src_arena, non_blocking=True),
                "h2d": lambda: dst_arena.copy_(host, non_blocking=True),
                "assemble": lambda: P.pallas_assemble_kv(st.dst, st.dst_tab[0], hdr, dst_arena, 1000, 1,
                                                         st.err)}
        times = {k: [] for k in legs}
        for it in range(reps + 2):
            evs = [torch.cuda.Event(enable_timing=True) for _ in range(len(legs) + 1)]
            evs[0].record(stream)
            for i, f in enumerate(legs.values()):
                f()
                evs[i + 1].record(stream)
            torch.cuda.synchronize()
            if it >= 2:
                for i, k in enumerate(legs):
                    times[k].append(evs[i].elapsed_time(evs[i + 1]))
        row = {"tokens": count, "bytes": nbytes}
        total = 0.0
        for k, v in times.items():
            ms = float(np.median(v))
            total += ms
            row[f"{k}_us"] = ms * 1e3
            row[f"{k}_payload_GBps"] = nbytes / ms / 1e6
        row["pcie_inclusive_GBps"] = nbytes / total / 1e6
        assert torch.equal(src_arena, dst_arena)
        out[name] = row
    torch.cuda.synchronize()
    assert int(st.err.item()) == 0
    return out


def overlapped_preparation(st, chunk=32, reps=3):
    """Prefix prefill on one stream while the suffix is assembled chunk by
    chunk (one launch per `chunk` tokens) on another: the time of each alone
    and of both together, from events on the two streams (median of
    `reps`)."""
    import numpy as np
    import torch

    P, cfg = st.P, st.cfg
    n, p = st.ns[0], st.ps[0]
    hdrs = [P.ChunkHeader(1000, 1, t, min(chunk, n - t), (t - p) * st.row_bytes, cfg.n_layers,
                          cfg.n_kv_heads, cfg.head_dim, 2) for t in range(p, n, chunk)]
    P.pallas_pack_suffix_blocks(st.src, st.src_tab[0], [P.ChunkDesc(h.start_pos, h.num_tokens, h.arena_offset)
                                                        for h in hdrs], st.arena, st.err)
    sa, sb = torch.cuda.Stream(), torch.cuda.Stream()

    def prefill():
        st.model.prefill_prefix(st.prefix_ids[:p], [0, p], st.dst_tab[:1], st.dst, st.ws, st.err, stream=sa)

    def assemble():
        for h in hdrs:
            P.pallas_assemble_kv(st.dst, st.dst_tab[0], [h], st.arena, 1000, 1, st.err, stream=sb)

    def timed(do_prefill, do_assemble):
        e = {k: torch.cuda.Event(enable_timing=True) for k in ("a0", "a1", "b0", "b1")}
        torch.cuda.synchronize()
        e["a0"].record(sa)
        e["b0"].record(sb)
        if do_prefill:
            prefill()
        if do_assemble:
            assemble()
        e["a1"].record(sa)
        e["b1"].record(sb)
        torch.cuda.synchronize()
        return e["a0"].elapsed_time(e["a1"]), e["b0"].elapsed_time(e["b1"])

    res = {"prefill_alone": [], "assemble_alone": [], "prefill_together": [], "assemble_together": []}
    timed(True, True)
    for _ in range(reps):
        res["prefill_alone"].append(timed(True, False)[0])
        res["assemble_alone"].append(timed(False, True)[1])
        a, b = timed(True, True)
        res["prefill_together"].append(a)
        res["assemble_together"].append(b)
    out = {k + "_ms": float(np.median(v)) for k, v in res.items()}
    out["chunks"] = len(hdrs)
    out["chunk_tokens"] = chunk
    out["prefill_slowdown"] = out["prefill_together_ms"] / out["prefill_alone_ms"]
    torch.cuda.synchronize()
    assert int(st.err.item()) == 0
    return out


def paced_preparation(st, rates_mbps=(100, 300, 500), chunk=32, prefills=6):
    """Overlapped preparation with the suffix arriving at network rates
    (the evaluation's links run at 100-500 Mbps): `prefills` back-to-back
    prefix prefills are enqueued on one stream (from a host thread), while
    the main thread releases one `chunk`-token chunk assembly on another
    stream each time a chunk's payload would have crossed a link of the
    given rate (payload bits / rate), until the prefills finish.  Reports,
    per rate, the chunks released, the median prefill time against the
    prefills alone, and the chunk assemblies' times (events around each
    launch on its stream: waiting for CU slots plus copying)."""
    import threading
    import numpy as np
    import torch

    P, cfg = st.P, st.cfg
    n, p = st.ns[0], st.ps[0]
    hdrs = [P.ChunkHeader(1000, 1, t, min(chunk, n - t), (t - p) * st.row_bytes, cfg.n_layers,
                          cfg.n_kv_heads, cfg.head_dim, 2) for t in range(p, n, chunk)]
    P.pallas_pack_suffix_blocks(st.src, st.src_tab[0], [P.ChunkDesc(h.start_pos, h.num_tokens, h.arena_offset)
                                                        for h in hdrs], st.arena, st.err)
    sa, sb = torch.cuda.Stream(), torch.cuda.Stream()
    chunk_bits = chunk * st.row_bytes * 8

    def run(rate):
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(prefills)]
        done = torch.cuda.Event()
        torch.cuda.synchronize()

        def enqueue():
            for a, b in evs:
                a.record(sa)
                st.model.prefill_prefix(st.prefix_ids[:p], [0, p], st.dst_tab[:1], st.dst, st.ws, st.err,
                                        stream=sa)
                b.record(sa)
            done.record(sa)

        th = threading.Thread(target=enqueue)
        t0 = time.perf_counter()
        th.start()
        asm = []
        if rate:
            interval = chunk_bits / (rate * 1e6)
            k = 0
            while True:
                target = t0 + (k + 1) * interval
                now = time.perf_counter()
                if now < target:
                    time.sleep(target - now)
                if not th.is_alive() and done.query():
                    break
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record(sb)
                P.pallas_assemble_kv(st.dst, st.dst_tab[0], [hdrs[k % len(hdrs)]], st.arena, 1000, 1, st.err,
                                     stream=sb)
                e1.record(sb)
                asm.append((e0, e1))
                k += 1
        th.join()
        torch.cuda.synchronize()
        return [a.elapsed_time(b) for a, b in evs], [a.elapsed_time(b) * 1e3 for a, b in asm]

    run(None)
    alone, _ = run(None)
    out = {"chunk_tokens": chunk, "chunk_bytes": chunk * st.row_bytes, "prefills": prefills,
           "prefill_alone_ms": float(np.median(alone)), "rows": []}
    for rate in rates_mbps:
        pre, asm = run(rate)
        row = {"rate_mbps": rate, "chunk_interval_ms": chunk_bits / (rate * 1e6) * 1e3,
               "chunks_released": len(asm), "prefill_ms": float(np.median(pre)),
               "prefill_slowdown": float(np.median(pre)) / out["prefill_alone_ms"]}
        if asm:
            row["assemble_us_median"] = float(np.median(asm))
            row["assemble_us_max"] = float(np.max(asm))
        out["rows"].append(row)
    torch.cuda.synchronize()
    assert int(st.err.item()) == 0
    return out


def scheduler_decision(P, cfg, prefix_tokens, prefill_ms, assemble_ms, decode_ms, calls=20000):
    """The Scheduler Engine fed with this run's measurements: r_p = the
    measured prefix-prefill rate, r_d = one token per measured decode step,
    T_0 = the measured assembly plus decode step, s_kv of the model; the
    goodput is the paper's representative 300 Mbps (context, not measured
    here), alpha 0.8, T_max 5 s, a 10 ms grid, 5 s predicted to handover.
    Reports the selected window and the mean time of one decision through
    the binding (ctypes call included)."""
    params = dict(r_p=prefix_tokens / (prefill_ms / 1e3), r_d=1e3 / decode_ms, goodput=300e6 / 8,
                  s_kv=float(cfg.s_kv), t_load=0.0, t_0=(assemble_ms + decode_ms) / 1e3, alpha=0.8,
                  t_max=5.0, dt=0.01)
    k_curr, t_remain = float(prefix_tokens), 5.0
    d = P.pallas_window_select(k_curr, t_remain, **params)
    t0 = time.perf_counter()
    for _ in range(calls):
        P.pallas_window_select(k_curr, t_remain, **params)
    us = (time.perf_counter() - t0) / calls * 1e6
    # The trade-off behind the choice (the shape of the paper's window
    # figures): the model's terms at windows from 0 to T_max.
    curve = []
    for t_w in sorted({0.0, 0.05, 0.1, 0.3, 0.5, 1.0, 2.0, 3.0, params["t_max"], d.t_w}):
        e = P.pallas_window_evaluate(k_curr, t_remain, t_w, **params)
        curve.append({"t_w": t_w, "cost": e.cost, "t_sit_s": e.t_sit, "t_early_s": e.t_early,
                      "t_hist_s": e.t_hist, "t_res_s": e.t_res, "l_hist": e.l_hist})
    return {"inputs": {**params, "k_curr": k_curr, "t_remain": t_remain}, "curve": curve,
            "t_w": d.t_w, "t_sit_s": d.t_sit, "t_early_s": d.t_early, "t_hist_s": d.t_hist,
            "t_res_s": d.t_res, "trigger": bool(d.trigger), "candidates": d.n_candidates,
            "decision_us": us}


def cpu_baseline(setup):
    """The oracle's first decoder layer (float64 numpy) over the workload's
    prefix rows, scaled by the layer count; plus the oracle's pack of the
    suffix from a host copy of the source pool and its assembly into a host
    copy of the target pool (GB/s = read + write of the payload)."""
    import numpy as np
    import torch
    from oracle import model as om
    from oracle import paged

    blas = "unknown"
    try:
        from threadpoolctl import threadpool_info
        infos = [i for i in threadpool_info() if i.get("user_api") == "blas"]
        threads = max([i.get("num_threads", 1) for i in infos] or [os.cpu_count() or 1])
        if infos:
            blas = f"{infos[0].get('internal_api', '?')} {infos[0].get('version', '')}".strip()
    except Exception:  # pragma: no cover
        threads = os.cpu_count() or 1
    cpu_model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    cpu_model = line.split(":", 1)[1].strip()
                    break
    except OSError:  # pragma: no cover
        pass
    cfg = setup.cfg
    shp = om.Shape.of(cfg)
    w = {k: v.to("cpu", torch.float64).numpy() for k, v in setup.layers[0].items()}
    i0 = 0
    p = setup.ps[i0]
    ids = setup.ids[i0][:p]
    r = setup.glob["embed"][torch.as_tensor(ids, dtype=torch.long, device="cuda")].to("cpu", torch.float64).numpy()
    pos = np.arange(p)
    t0 = time.perf_counter()
    om.layer(r, pos, None, None, w, shp, om.bf16_round)
    t_layer = time.perf_counter() - t0
    tok_s = p / (t_layer * cfg.n_layers)
    # pack of the first request's suffix
    n = setup.ns[i0]
    src = setup.src.view(torch.int16).cpu().numpy()
    bt = setup.src_tab[i0].cpu().numpy()
    t0 = time.perf_counter()
    chunk = paged.pack(src, bt, p, n - p)
    t_pack = time.perf_counter() - t0
    del src
    # assembly of that chunk into a host copy of the target pool
    dst = setup.dst.view(torch.int16).cpu().numpy()
    dbt = setup.dst_tab[i0].cpu().numpy()
    hdr = paged.ChunkHeader(1, 1, p, n - p, cfg.n_layers, cfg.n_kv_heads, cfg.head_dim, 2)
    t0 = time.perf_counter()
    paged.assemble(dst, dbt, [hdr], [chunk], 1, 1)
    t_asm = time.perf_counter() - t0
    del dst
    return {
        "value": tok_s, "unit": "tokens/s", "cores": int(threads), "kind": "oracle",
        "cpu_model": cpu_model, "blas": blas, "host_cpus": os.cpu_count(),
        "sample": (f"oracle decoder layer 0 in float64 over the {p}-token prefix "
                   f"({t_layer:.2f} s), scaled by {cfg.n_layers} layers"),
        "pack_GBps": 2 * chunk.nbytes / t_pack / 1e9,
        "pack_sample": f"oracle pack of the {n - p}-token suffix ({chunk.nbytes / 1e6:.0f} MB) on 1 thread",
        "assemble_GBps": 2 * chunk.nbytes / t_asm / 1e9,
        "assemble_sample": f"oracle assembly of that chunk into a host copy of the target pool on 1 thread",
    }


def copy_roofline(kind, phase_ms, copy_bytes, suffix_tokens, prof):
    """Pack or assemble against the HBM peak: algorithmic bytes (payload read
    + written) over the phase's time in the timed steps, the average launch
    time from the profiled pass, and the counter-measured traffic per launch
    where it was taken."""
    ms, n = prof.get(kind, (0.0, 0))
    traffic = copy_traffic_bytes(kind, suffix_tokens)
    gbps = copy_bytes / (phase_ms / 1e3) / 1e9
    return {"bound": "hbm", "bytes": copy_bytes, "ms": phase_ms, "achieved": gbps,
            "peak": PEAK_HBM_GBPS, "unit": "GB/s", "frac": gbps / PEAK_HBM_GBPS,
            "kernel_avg_us": ms / n * 1e3 if n else None,
            "traffic": traffic,
            "traffic_ratio": traffic / copy_bytes if traffic else None}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not supported "
              "(the reconstruction path runs on one GPU with no collectives).", file=sys.stderr)
        sys.exit(2)
    if args.copy_calibration:
        copy_calibration()
        return
    import torch
    from workloads import workload

    P = load_library()
    wl = workload(args.workload)
    cfg = wl.model
    print(f"[bench] workload {wl.name}: {cfg.n_layers} layers, hidden {cfg.hidden}, "
          f"{cfg.n_q_heads}/{cfg.n_kv_heads} heads, d {cfg.head_dim}, ffn {cfg.ffn}, "
          f"ctx {wl.ctx}, prefix {wl.prefix}", file=sys.stderr, flush=True)
    t0 = time.time()
    st = Setup(P, wl, args.seed)
    print(f"[bench] setup {time.time() - t0:.1f} s", file=sys.stderr, flush=True)

    stream = torch.cuda.current_stream()
    phases = ("prefill", "pack", "assemble", "decode")
    fns = (st.prefill, st.pack, st.assemble, st.decode)

    def step(ev=None):
        for k, f in enumerate(fns):
            if ev is not None:
                ev[k].record(stream)
            f()
        if ev is not None:
            ev[len(fns)].record(stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    print("[bench] warmup done", file=sys.stderr, flush=True)

    # Timed steps: the library records events only around the roofline
    # kernel's launches (the gate|up GEMM), on the stream it launches on.
    P.pallas_profile_reset()
    P.pallas_profile_enable(["gemm_gate_up"])
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(len(fns) + 1)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t_start = torch.cuda.Event(enable_timing=True)
    t_end = torch.cuda.Event(enable_timing=True)
    wall0 = time.perf_counter()
    t_start.record(stream)
    for k in range(args.steps):
        step(evs[k])
    t_end.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    roof_ms, roof_n = P.pallas_profile_read()["gemm_gate_up"]
    roof_ghz, roof_wgs = P.pallas_profile_clock("gemm_gate_up")
    assert int(st.err.item()) == 0, "device-side error flag raised"
    # The same number of steps again with events around every launch:
    # per-class averages for the breakdown.
    P.pallas_profile_reset()
    P.pallas_profile_enable(P.KERNEL_CLASSES)
    p_start = torch.cuda.Event(enable_timing=True)
    p_end = torch.cuda.Event(enable_timing=True)
    p_start.record(stream)
    for k in range(args.steps):
        step()
    p_end.record(stream)
    torch.cuda.synchronize()
    prof = P.pallas_profile_read()
    gemm_sclk = {k: P.pallas_profile_clock(k)[0] for k in ("gemm_qkv", "gemm_o", "gemm_gate_up", "gemm_down")}
    ms_step_profiled = p_start.elapsed_time(p_end) / args.steps
    P.pallas_profile_enable([])
    assert int(st.err.item()) == 0, "device-side error flag raised"

    ms_step = t_start.elapsed_time(t_end) / args.steps
    phase_ms = {ph: sum(evs[k][i].elapsed_time(evs[k][i + 1]) for k in range(args.steps)) / args.steps
                for i, ph in enumerate(phases)}
    prefix_tokens = sum(st.ps)
    flops = sum(cfg.prefill_flops(p) for p in st.ps)
    copy_bytes = 2 * st.suffix_tokens * cfg.s_kv     # read + write of the payload
    value = prefix_tokens / (ms_step / 1e3)

    gu_avg_s = roof_ms / roof_n / 1e3
    gu_flops = 2.0 * prefix_tokens * 2 * cfg.ffn * cfg.hidden
    achieved = gu_flops / gu_avg_s / 1e12
    kernels = {k: {"avg_us": v[0] / v[1] * 1e3, "launches_per_step": v[1] / args.steps}
               for k, v in prof.items() if v[1]}
    for k, ghz in gemm_sclk.items():
        if k in kernels and ghz > 0:
            kernels[k]["sclk_ghz"] = ghz

    out = {
        "metric": METRIC,
        "value": value,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": (f"{wl.name}: {cfg.n_layers}-layer decoder, hidden {cfg.hidden}, "
                         f"{cfg.n_q_heads}/{cfg.n_kv_heads} heads, head_dim {cfg.head_dim}, "
                         f"ffn {cfg.ffn}, vocab {cfg.vocab}, qk_norm {cfg.qk_norm}; "
                         f"{wl.num_seqs} request(s), ctx {wl.ctx}, prefix {wl.prefix}, "
                         f"suffix chunks of {wl.chunk_tokens or 'the whole suffix'} tokens, page 16"),
            "step": "prefix prefill + suffix pack + assembly + one decode step",
            "prefix_tokens": prefix_tokens,
            "suffix_tokens": st.suffix_tokens,
        },
        "breakdown": {
            "prefill_ms": phase_ms["prefill"],
            "prefill_tokens_per_s": prefix_tokens / (phase_ms["prefill"] / 1e3),
            "prefill_tflops": flops / (phase_ms["prefill"] / 1e3) / 1e12,
            "prefill_mfma_frac": flops / (phase_ms["prefill"] / 1e3) / 1e12 / PEAK_BF16_TFLOPS,
            "pack_ms": phase_ms["pack"],
            "pack_GBps": copy_bytes / (phase_ms["pack"] / 1e3) / 1e9,
            "pack_hbm_frac": copy_bytes / (phase_ms["pack"] / 1e3) / 1e9 / PEAK_HBM_GBPS,
            "assemble_ms": phase_ms["assemble"],
            "assemble_GBps": copy_bytes / (phase_ms["assemble"] / 1e3) / 1e9,
            "assemble_hbm_frac": copy_bytes / (phase_ms["assemble"] / 1e3) / 1e9 / PEAK_HBM_GBPS,
            "decode_ms": phase_ms["decode"],
            "kernels": kernels,
            "ms_per_step_with_kernel_events": ms_step_profiled,
            "host_wall_s": wall,
        },
        "roofline": {
            "bound": "mfma",
            "kernel": "gemm_bf16_kernel<2> (gate|up projection + SwiGLU)",
            "achieved": achieved,
            "peak": PEAK_BF16_TFLOPS,
            "unit": "TFLOP/s",
            "frac": achieved / PEAK_BF16_TFLOPS,
            # Shader clock measured inside the same launches (per-workgroup
            # clock and wall-clock counters); the peak assumes 2.4 GHz.
            "sclk_ghz": roof_ghz,
            "frac_clock_adjusted": (achieved / (PEAK_BF16_TFLOPS * roof_ghz / NOMINAL_SCLK_GHZ)
                                    if roof_ghz > 0 else None),
            "traffic": gemm_traffic_bytes(),
            "algorithmic_bytes": 2.0 * (prefix_tokens * cfg.hidden + 2 * cfg.ffn * cfg.hidden
                                        + prefix_tokens * cfg.ffn),
            # The two halves of the metric, each against its own roofline:
            # the whole prefix prefill (every kernel of the phase) against
            # the bf16 MFMA peak, and pack / assemble of the suffix payload
            # (read once + written once) against the HBM peak.
            "prefill_whole": {
                "bound": "mfma", "flops": flops, "ms": phase_ms["prefill"],
                "achieved": flops / (phase_ms["prefill"] / 1e3) / 1e12, "peak": PEAK_BF16_TFLOPS,
                "unit": "TFLOP/s",
                "frac": flops / (phase_ms["prefill"] / 1e3) / 1e12 / PEAK_BF16_TFLOPS,
            },
            "pack": copy_roofline("pack", phase_ms["pack"], copy_bytes, st.suffix_tokens, prof),
            "assemble": copy_roofline("assemble", phase_ms["assemble"], copy_bytes, st.suffix_tokens, prof),
        },
        "cpu_baseline": None,
    }
    if not args.no_chunked:
        print("[bench] chunked prefill", file=sys.stderr, flush=True)
        out["chunked_prefill"] = chunked_prefill(st)
        out["chunked_prefill"]["whole_prefix_ms"] = phase_ms["prefill"]
        print("[bench] post-handover recompute", file=sys.stderr, flush=True)
        out["post_handover_recompute"] = post_handover_recompute(st, phase_ms["assemble"])
    out["scheduler"] = scheduler_decision(P, cfg, st.ps[0] if wl.num_seqs == 1 else prefix_tokens,
                                          phase_ms["prefill"], phase_ms["assemble"], phase_ms["decode"])
    if not args.no_staging:
        print("[bench] wire staging and overlapped preparation", file=sys.stderr, flush=True)
        out["wire_staging"] = wire_staging(st)
        out["overlapped_preparation"] = overlapped_preparation(st)
        out["paced_preparation"] = paced_preparation(st)
    if not args.no_stress:
        print("[bench] stress-layout copies", file=sys.stderr, flush=True)
        out["copies_stress"] = copies_stress(P, args.seed)
    if not args.no_cpu_baseline:
        print("[bench] timing the CPU oracle sample", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(st)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
