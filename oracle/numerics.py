"""bf16 rounding for the oracle.

The KV cache holds 2-byte elements (Section 2.1, Eq. 1 with b = 2), and the
decoders the paper serves run in bf16.  The oracle computes in float64 and
rounds to bf16 (round to nearest, ties to even, 8 significant bits) at the
points where the model stores a bf16 tensor.
"""
import numpy as np

_MIN_NORMAL_EXP = -125   # frexp exponent of 2**-126, bf16's smallest normal


def bf16_round(x) -> np.ndarray:
    """Round float64 values to the nearest bf16 value (ties to even)."""
    x = np.asarray(x, dtype=np.float64)
    _, e = np.frexp(x)
    e = np.maximum(e, _MIN_NORMAL_EXP)
    ulp = np.ldexp(1.0, e - 8)
    return np.rint(x / ulp) * ulp


def bf16_round_as(x) -> np.ndarray:
    """bf16 rounding that keeps the input's floating type (for forwards
    evaluated in float32)."""
    x = np.asarray(x)
    return bf16_round(x.astype(np.float64)).astype(x.dtype)


def no_round(x) -> np.ndarray:
    """Identity rounding: the same forward in plain float64."""
    return np.asarray(x, dtype=np.float64)


def bf16_bits(x) -> np.ndarray:
    """bf16 bit patterns (uint16) of values that are exactly bf16."""
    f = np.asarray(x, dtype=np.float32)
    return (f.view(np.uint32) >> 16).astype(np.uint16)


def from_bf16_bits(bits) -> np.ndarray:
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    return b.view(np.float32).astype(np.float64)
