"""The whole reconstruction of one workload on the GPU, for the full-size and
reduced-depth parity tests: the source's full prefill of every request, the
pack of each suffix (in the workload's chunk size), the target's varlen
prefix prefill, the assembly of the chunks and one batched decode step over
the assembled caches, plus layer-local oracle checks of sampled layers
(``check_prefill_layer``, ``check_decode``).  Test glue: none of the
method's arithmetic is here; the oracle supplies the references."""
import numpy as np
import torch

from helpers import (TOL, LazyOracleLayers, check_layer_local, rel_err, residual_rows, to_np64,
                     truncated_model)
from oracle import model as om
from workloads import gen

DEV = "cuda"


class Recon:
    """Source full prefill, pack, target prefix prefill, assembly, decode."""

    def __init__(self, P, wl, seed=0):
        self.P, self.wl, cfg = P, wl, wl.model
        self.cfg = cfg
        self.glob, self.layers = gen.model_weights(cfg, seed=seed, device=DEV)
        self.model = P.Model(cfg, self.glob, self.layers)
        self.ns, self.ps = list(wl.ctx), list(wl.prefix)
        B = len(self.ns)
        self.ids = [gen.token_ids(n + 1, cfg.vocab, seed=seed, stream=i).numpy()
                    for i, n in enumerate(self.ns)]
        pages = [wl.pages_for(n + 1) for n in self.ns]
        self.max_pages = max(pages)
        self.tot = tot = sum(pages)
        self.src_tab = torch.tensor(gen.disjoint_block_tables(pages, tot, self.max_pages, seed, 1),
                                    dtype=torch.int32, device=DEV)
        self.dst_tab = torch.tensor(gen.disjoint_block_tables(pages, tot, self.max_pages, seed, 2),
                                    dtype=torch.int32, device=DEV)
        shape = (cfg.n_layers, 2, tot, 16, cfg.n_kv_heads, cfg.head_dim)
        self.src = torch.zeros(shape, dtype=torch.bfloat16, device=DEV)
        self.dst = torch.zeros(shape, dtype=torch.bfloat16, device=DEV)
        self.err = torch.zeros(1, dtype=torch.int32, device=DEV)
        ws = self.model.workspace(max(sum(self.ps), max(self.ns)), B)
        for i, n in enumerate(self.ns):
            self.model.prefill_prefix(torch.tensor(self.ids[i][:n], dtype=torch.int32, device=DEV), [0, n],
                                      self.src_tab[i:i + 1], self.src, ws, self.err)
        self.cu = [0]
        for p in self.ps:
            self.cu.append(self.cu[-1] + p)
        self.prefix_ids = torch.tensor(np.concatenate([x[:p] for x, p in zip(self.ids, self.ps)]),
                                       dtype=torch.int32, device=DEV)
        self.model.prefill_prefix(self.prefix_ids, self.cu, self.dst_tab, self.dst, ws, self.err)
        del ws
        row = 2 * cfg.n_layers * cfg.n_kv_heads * cfg.head_dim * 2
        for i, (n, p) in enumerate(zip(self.ns, self.ps)):
            step = wl.chunk_tokens or (n - p)
            pieces = [(t, min(step, n - t)) for t in range(p, n, step)]
            offs = np.cumsum([0] + [c * row for _, c in pieces])
            arena = torch.empty(int(offs[-1]), dtype=torch.uint8, device=DEV)
            P.pallas_pack_suffix_blocks(self.src, self.src_tab[i],
                                        [P.ChunkDesc(s, c, int(o)) for (s, c), o in zip(pieces, offs)],
                                        arena, self.err)
            hdrs = [P.ChunkHeader(7 + i, 3, s, c, int(o), cfg.n_layers, cfg.n_kv_heads, cfg.head_dim, 2)
                    for (s, c), o in zip(pieces, offs)]
            assert P.pallas_check_coverage(p, [h.start_pos for h in hdrs], [h.num_tokens for h in hdrs], n) == 0
            P.pallas_assemble_kv(self.dst, self.dst_tab[i], hdrs, arena, 7 + i, 3, self.err)
            torch.cuda.synchronize()
            del arena
        self.tokens = torch.tensor([x[n] for x, n in zip(self.ids, self.ns)], dtype=torch.int32, device=DEV)
        self.logits_dst = torch.empty((B, cfg.vocab), dtype=torch.float32, device=DEV)
        self.logits_src = torch.empty((B, cfg.vocab), dtype=torch.float32, device=DEV)
        wsd = self.model.workspace(B, B)
        self.model.decode_step(self.tokens, self.ns, self.src_tab, self.src, self.logits_src, wsd, self.err)
        self.model.decode_step(self.tokens, self.ns, self.dst_tab, self.dst, self.logits_dst, wsd, self.err)
        torch.cuda.synchronize()
        # the residual leaving the last layer of the decode over the assembled caches
        self.r_final = residual_rows(wsd, B, cfg.hidden).double().cpu().numpy()
        del wsd
        assert int(self.err.item()) == 0
        self.lazy = LazyOracleLayers(self.layers)
        self.shp = om.Shape.of(cfg)
        self._inputs = {}

    def kv(self, pool, tab, i, n, layer):
        """[2, n, Hkv, d] float64 of one layer through one table."""
        page = 16
        t = np.arange(n)
        bt = tab[i].cpu().numpy()
        pages = torch.as_tensor(bt[t // page], device=DEV, dtype=torch.long)
        slots = torch.as_tensor(t % page, device=DEV, dtype=torch.long)
        return pool[layer, :, pages, slots].to(torch.float64).cpu().numpy()

    def check_properties(self):
        for i, (n, p) in enumerate(zip(self.ns, self.ps)):
            for l in range(self.cfg.n_layers):
                a = self.kv(self.dst, self.dst_tab, i, n, l)
                b = self.kv(self.src, self.src_tab, i, n, l)
                # prefix: target prefill == source prefill (causality), bitwise
                # suffix: assembled copy, bitwise
                np.testing.assert_array_equal(a, b, err_msg=f"request {i} layer {l}")
        assert torch.equal(self.logits_dst, self.logits_src)
        assert torch.isfinite(self.logits_dst).all()

    # -------------------------------------------------- layer-local inputs
    def prefill_input(self, l):
        """[M, H] float64: the residual the target's prefix prefill feeds
        layer l (rows in the call's order).  A model over layers [0, l]
        prefills the same ids into a scratch pool; its last layer runs only
        the K/V projection, so the workspace then holds layer l's input.
        Its layer-l K/V must equal the full model's bit for bit."""
        if l in self._inputs:
            return self._inputs[l]
        cfg, M = self.cfg, self.cu[-1]
        sub = truncated_model(self.P, cfg, self.glob, self.layers, l + 1)
        pool = torch.zeros((l + 1, 2, self.tot, 16, cfg.n_kv_heads, cfg.head_dim), dtype=torch.bfloat16,
                           device=DEV)
        ws = sub.workspace(M, len(self.ps))
        sub.prefill_prefix(self.prefix_ids, self.cu, self.dst_tab, pool, ws, self.err)
        torch.cuda.synchronize()
        r = residual_rows(ws, M, cfg.hidden).double().cpu().numpy()
        for i, p in enumerate(self.ps):
            np.testing.assert_array_equal(self.kv(pool, self.dst_tab, i, p, l),
                                          self.kv(self.dst, self.dst_tab, i, p, l))
        del pool, ws, sub
        self._inputs[l] = r
        return r

    def check_prefill_layer(self, l, tail=None):
        last = l == self.cfg.n_layers - 1
        r_in = self.prefill_input(l)
        r_next = None if last else self.prefill_input(l + 1)
        got = [self.kv(self.dst, self.dst_tab, i, p, l) for i, p in enumerate(self.ps)]
        w = self.lazy[l]
        worst = check_layer_local(r_in, self.cu, w, self.shp, [g[0] for g in got], [g[1] for g in got],
                                  r_next=r_next, tail=tail, label=f"layer {l}")
        print(f"layer {l}: K {worst[0]:.2e} V {worst[1]:.2e} residual update {worst[2]:.2e}")

    def decode_io(self, n_layers):
        """[B, H] float64: the residual leaving the last layer of a decode
        step by a model over layers [0, n_layers) on the assembled caches
        (the first n_layers layers of the target pool; the step rewrites
        the same K/V into slot n_i of those layers)."""
        if n_layers == self.cfg.n_layers:
            return self.r_final
        cfg, B = self.cfg, len(self.ns)
        sub = truncated_model(self.P, cfg, self.glob, self.layers, n_layers)
        logits = torch.empty((B, cfg.vocab), dtype=torch.float32, device=DEV)
        ws = sub.workspace(B, B)
        sub.decode_step(self.tokens, self.ns, self.dst_tab, self.dst[:n_layers], logits, ws, self.err)
        torch.cuda.synchronize()
        return residual_rows(ws, B, cfg.hidden).double().cpu().numpy()

    def check_decode(self, layers):
        """Final norm + lm_head on the GPU decode's final residual, and the
        oracle's decode layer l from the GPU's input to it over the GPU's
        cache of layer l, for l in ``layers``."""
        g = {k: to_np64(self.glob[k]) for k in ("final_norm", "lm_head")}
        ref = om.logits(self.r_final, g, self.shp)
        for i in range(len(self.ns)):
            e = rel_err(self.logits_dst[i].double().cpu().numpy(), ref[i])
            assert e <= TOL, f"request {i}: logits {e:.3g}"
        del g
        emb = to_np64(self.glob["embed"][self.tokens.long()])
        for l in layers:
            r_in = emb if l == 0 else self.decode_io(l)
            r_out = self.decode_io(l + 1)
            w = self.lazy[l]
            for i, n in enumerate(self.ns):
                kv = self.kv(self.dst, self.dst_tab, i, n + 1, l)
                ro, k, v = om.layer(r_in[i:i + 1], np.array([n]), kv[0, :n], kv[1, :n], w, self.shp, om.bf16_round)
                ek, ev = rel_err(kv[0, n], k[0]), rel_err(kv[1, n], v[0])
                eu = rel_err(r_out[i] - r_in[i], ro[0] - r_in[i])
                print(f"decode layer {l} request {i} at {n}: K {ek:.2e} V {ev:.2e} residual update {eu:.2e}")
                assert ek <= TOL and ev <= TOL and eu <= TOL, f"decode layer {l} request {i}"
