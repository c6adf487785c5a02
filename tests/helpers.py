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
