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
