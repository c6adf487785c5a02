"""Test-side glue: turn generated torch tensors into the numpy inputs the
oracle takes.  Holds none of the method's arithmetic."""
import numpy as np
import torch

from oracle.model import Shape


def to_np64(t: torch.Tensor) -> np.ndarray:
    return t.detach().to("cpu", torch.float64).numpy()


def oracle_weights(glob, layers):
    g = {k: to_np64(v) for k, v in glob.items()}
    ls = [{k: to_np64(v) for k, v in l.items()} for l in layers]
    return g, ls


def shape_of(cfg) -> Shape:
    return Shape.of(cfg)


def bits(t: torch.Tensor) -> np.ndarray:
    """uint16 bit patterns of a bf16 tensor."""
    return t.detach().cpu().contiguous().view(torch.int16).numpy().view(np.uint16)


# ------------------------------------------------------------ library access
def ensure_lib():
    """Load the built HIP library, building it first only if it is absent."""
    import os
    import paper_2608_16477_amd as P
    if not os.path.exists(P.library_path()):
        from paper_2608_16477_amd import build
        build.build()
    P.lib()
    return P


def pool_np_bits(pool: torch.Tensor) -> np.ndarray:
    return bits(pool)


def make_headers(P, pieces, cfg_kv, req=1, epoch=1):
    """pieces: list of (start, count, arena_offset)."""
    L, hkv, d = cfg_kv
    return [P.ChunkHeader(req, epoch, s, c, off, L, hkv, d, 2) for s, c, off in pieces]


# ------------------------------------------------------------ reconstruction
def gpu_model(P, cfg, glob, layers, device="cuda"):
    g = {k: v.to(device).contiguous() for k, v in glob.items()}
    ls = [{k: v.to(device).contiguous() for k, v in l.items()} for l in layers]
    return P.Model(cfg, g, ls)


def empty_pool(cfg, pages, device="cuda", fill_bits=None):
    shape = (cfg.n_layers, 2, pages, cfg.page_size, cfg.n_kv_heads, cfg.head_dim)
    pool = torch.empty(shape, dtype=torch.bfloat16, device=device)
    if fill_bits is not None:
        pool.view(torch.int16).fill_(fill_bits)
    return pool


def kv_logical(pool: torch.Tensor, bt: np.ndarray, n: int) -> np.ndarray:
    """[L, 2, n, Hkv, d] float64 values of positions [0, n) through table bt."""
    page = pool.shape[3]
    t = np.arange(n)
    pages = torch.as_tensor(np.asarray(bt)[t // page], device=pool.device, dtype=torch.long)
    slots = torch.as_tensor(t % page, device=pool.device, dtype=torch.long)
    return pool[:, :, pages, slots].to(torch.float64).cpu().numpy()


def rel_err(got: np.ndarray, ref: np.ndarray) -> float:
    return float(np.max(np.abs(got - ref)) / max(np.max(np.abs(ref)), 1e-30))


TOL = 1e-2   # max|gpu - ref| <= TOL * max|ref| per (layer, K|V) tensor and per logits row


class LazyOracleLayers:
    """Per-layer float64 numpy weights, converted from device tensors on
    access and kept only for the most recent layer (full-size models do not
    fit in host memory at float64)."""

    def __init__(self, layers):
        self.layers = layers
        self._cache = (None, None)

    def __len__(self):
        return len(self.layers)

    def __getitem__(self, l):
        if self._cache[0] != l:
            self._cache = (l, {k: to_np64(v) for k, v in self.layers[l].items()})
        return self._cache[1]


def oracle_globals(glob, need_embed_rows=None):
    """Float64 globals; the embedding is gathered to the rows needed."""
    g = {k: to_np64(v) for k, v in glob.items() if k not in ("embed", "lm_head")}
    return g


# ------------------------------------------------------------ layer-local parity
def residual_rows(ws: torch.Tensor, rows: int, hidden: int) -> torch.Tensor:
    """The residual section of a workspace (pallas.h, pallas_workspace_size):
    float32 [rows][hidden].  After a prefill it holds the residual entering
    the model's last layer, after a decode the residual leaving it."""
    return ws[: rows * hidden * 4].view(torch.float32).view(rows, hidden)


def truncated_model(P, cfg, glob, layers, n_layers):
    """A model handle over the first ``n_layers`` layers of a model (the same
    device weight tensors)."""
    return P.Model(cfg.replace(n_layers=n_layers), glob, layers[:n_layers])


def check_layer_local(r_in, cu, w, shp, got_k, got_v, r_next=None, tail=None, kv_only=False,
                      label=""):
    """Layer-local oracle parity of one decoder layer of a prefill.

    ``r_in [M, H]`` is the residual the GPU fed the layer (float64 of its
    float32 values), rows of sequence i at ``[cu[i], cu[i+1])`` and
    positions 0, 1, ...  The oracle runs the layer from that input.  Its K
    and V of every position must match ``got_k[i], got_v[i] [p_i, Hkv, d]``
    (the GPU's K/V of the layer) within TOL max|ref| per sequence and
    tensor.  With ``r_next`` (the GPU's residual leaving the layer), the
    update the layer adds, r_next - r_in, must match the oracle's within TOL
    of its max, on every row or on the last ``tail`` rows of each sequence
    (their attention then reads the oracle's K/V of the earlier rows).
    Returns the largest relative errors (K, V, update)."""
    from oracle import model as om
    worst = [0.0, 0.0, 0.0]
    for i in range(len(cu) - 1):
        a, b = cu[i], cu[i + 1]
        x = r_in[a:b]
        pos = np.arange(b - a)
        full = r_next is not None and tail is None
        r_out, k, v = om.layer(x, pos, None, None, w, shp, om.bf16_round, kv_only=not full)
        ek, ev = rel_err(got_k[i], k), rel_err(got_v[i], v)
        worst[0], worst[1] = max(worst[0], ek), max(worst[1], ev)
        assert ek <= TOL and ev <= TOL, f"{label} sequence {i}: K {ek:.3g}, V {ev:.3g}"
        if r_next is None or kv_only:
            continue
        s = 0 if tail is None else max(0, (b - a) - tail)
        if not full:
            r_out, _, _ = om.layer(x[s:], pos[s:], k[:s] if s else None, v[:s] if s else None, w, shp,
                                   om.bf16_round)
        eu = rel_err(r_next[a + s:b] - x[s:], r_out - x[s:])
        worst[2] = max(worst[2], eu)
        assert eu <= TOL, f"{label} sequence {i}: residual update {eu:.3g}"
    return worst
