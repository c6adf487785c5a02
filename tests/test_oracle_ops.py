"""Oracle pins for the per-token operations: bf16 rounding, RMSNorm, rotary
embedding, SiLU and causal grouped-query attention.  Each is checked against
something other than itself: a library routine on a special case, a closed
form, an invariant, or brute force on tiny inputs."""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import model as om
from oracle import numerics as on

RNG = np.random.default_rng(1234)


# ---------------------------------------------------------------- bf16 rounding
def test_bf16_round_matches_torch_on_float32_inputs():
    x = RNG.standard_normal(200000).astype(np.float32) * np.float32(3.0)
    # add exact ties: values halfway between two bf16 neighbours
    base = (RNG.standard_normal(1000).astype(np.float32).view(np.uint32) & 0xFFFF0000)
    ties = (base | 0x8000).view(np.float32)
    x = np.concatenate([x, ties, np.float32([0.0, -0.0, 1.0, 2**-130, 3.0e38])])
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    got = on.bf16_round(x.astype(np.float64))
    np.testing.assert_array_equal(got, ref)


def test_bf16_round_ties_to_even_and_idempotent():
    one = 1.0
    ulp = 2.0 ** -7
    assert on.bf16_round(one + ulp / 2) == one            # tie -> even (1.0)
    assert on.bf16_round(one + 3 * ulp / 2) == one + 2 * ulp
    x = RNG.standard_normal(1000)
    r = on.bf16_round(x)
    np.testing.assert_array_equal(on.bf16_round(r), r)
    np.testing.assert_array_equal(on.from_bf16_bits(on.bf16_bits(r)), r)
    assert np.all(np.abs(r - x) <= np.abs(x) * 2.0 ** -8)


# ---------------------------------------------------------------- RMSNorm
def test_rmsnorm_matches_torch():
    x = RNG.standard_normal((7, 96))
    g = 1 + 0.1 * RNG.standard_normal(96)
    ref = F.rms_norm(torch.from_numpy(x), (96,), torch.from_numpy(g), eps=1e-6).numpy()
    np.testing.assert_allclose(om.rmsnorm(x, g, 1e-6), ref, rtol=1e-12, atol=1e-12)


def test_rmsnorm_scale_invariant_and_unit_rms():
    x = RNG.standard_normal((5, 64)) * 3
    g = np.ones(64)
    y = om.rmsnorm(x, g, 0.0)
    np.testing.assert_allclose(np.sqrt(np.mean(y * y, axis=-1)), 1.0, rtol=1e-12)
    np.testing.assert_allclose(om.rmsnorm(7.5 * x, g, 0.0), y, rtol=1e-12)


# ---------------------------------------------------------------- RoPE
def test_rope_identity_at_position_zero():
    x = RNG.standard_normal((1, 3, 64))
    np.testing.assert_array_equal(om.rope(x, np.array([0]), 1e6), x)


def test_rope_matches_complex_rotation():
    """Half-split rotary embedding is multiplication of (x_i + j x_{i+d/2})
    by exp(j * pos * theta^(-2i/d))."""
    d, theta = 64, 1e4
    x = RNG.standard_normal((5, 2, d))
    pos = np.array([0, 1, 7, 100, 4095])
    z = x[..., : d // 2] + 1j * x[..., d // 2:]
    freqs = np.array([theta ** (-2.0 * i / d) for i in range(d // 2)])
    rot = np.exp(1j * pos[:, None, None] * freqs[None, None, :])
    w = z * rot
    ref = np.concatenate([w.real, w.imag], axis=-1)
    np.testing.assert_allclose(om.rope(x, pos, theta), ref, rtol=1e-12, atol=1e-12)


def test_rope_relative_position_property():
    d = 128
    q = RNG.standard_normal((1, 1, d))
    k = RNG.standard_normal((1, 1, d))
    def dot(m, n):
        return float(np.sum(om.rope(q, np.array([m]), 1e6) * om.rope(k, np.array([n]), 1e6)))
    assert abs(dot(10, 3) - dot(107, 100)) < 1e-9
    assert abs(dot(5, 5) - float(np.sum(q * k))) < 1e-9
    # pair norms preserved
    y = om.rope(q, np.array([33]), 1e6)
    n0 = q[..., :64] ** 2 + q[..., 64:] ** 2
    n1 = y[..., :64] ** 2 + y[..., 64:] ** 2
    np.testing.assert_allclose(n1, n0, rtol=1e-12)


# ---------------------------------------------------------------- SiLU
def test_silu():
    assert om.silu(np.array([0.0]))[0] == 0.0
    x = RNG.standard_normal(100) * 5
    np.testing.assert_allclose(om.silu(x), F.silu(torch.from_numpy(x)).numpy(), rtol=1e-12)


# ---------------------------------------------------------------- attention
def brute_attention(q, q_pos, k, v):
    T, Hq, d = q.shape
    S, Hkv, _ = k.shape
    G = Hq // Hkv
    out = np.zeros((T, Hq, d))
    for t in range(T):
        for h in range(Hq):
            kh = h // G
            w = []
            for j in range(S):
                if j <= q_pos[t]:
                    w.append(math.exp(sum(q[t, h, i] * k[j, kh, i] for i in range(d)) / math.sqrt(d)))
                else:
                    w.append(0.0)
            z = sum(w)
            for i in range(d):
                out[t, h, i] = sum(w[j] * v[j, kh, i] for j in range(S)) / z
    return out


def test_attention_brute_force_gqa():
    T, Hq, Hkv, d = 6, 4, 2, 8
    q = RNG.standard_normal((T, Hq, d))
    k = RNG.standard_normal((T, Hkv, d))
    v = RNG.standard_normal((T, Hkv, d))
    pos = np.arange(T)
    np.testing.assert_allclose(om.causal_attention(q, pos, k, v),
                               brute_attention(q, pos, k, v), rtol=1e-10, atol=1e-12)


def test_attention_decode_row_brute_force():
    """A single query at position 5 over 6 cached keys (the decode shape)."""
    Hq, Hkv, d = 6, 3, 4
    q = RNG.standard_normal((1, Hq, d))
    k = RNG.standard_normal((6, Hkv, d))
    v = RNG.standard_normal((6, Hkv, d))
    pos = np.array([5])
    np.testing.assert_allclose(om.causal_attention(q, pos, k, v),
                               brute_attention(q, pos, k, v), rtol=1e-10, atol=1e-12)


def test_attention_special_cases():
    T, Hq, Hkv, d = 9, 4, 1, 16
    q = RNG.standard_normal((T, Hq, d))
    v = RNG.standard_normal((T, Hkv, d))
    k = RNG.standard_normal((T, Hkv, d))
    out = om.causal_attention(q, np.arange(T), k, v)
    # position 0 sees only itself
    for h in range(Hq):
        np.testing.assert_allclose(out[0, h], v[0, 0], rtol=1e-14)
    # identical keys: uniform weights, the running mean of V
    ksame = np.repeat(k[:1], T, axis=0)
    out2 = om.causal_attention(q, np.arange(T), ksame, v)
    run_mean = np.cumsum(v[:, 0], axis=0) / np.arange(1, T + 1)[:, None]
    for h in range(Hq):
        np.testing.assert_allclose(out2[:, h], run_mean, rtol=1e-12, atol=1e-14)


@pytest.mark.parametrize("Hq,Hkv", [(4, 4), (8, 2), (6, 3)])
def test_attention_matches_torch_sdpa(Hq, Hkv):
    T, d = 33, 32
    q = RNG.standard_normal((T, Hq, d))
    k = RNG.standard_normal((T, Hkv, d))
    v = RNG.standard_normal((T, Hkv, d))
    tq = torch.from_numpy(q).permute(1, 0, 2)[None]
    tk = torch.from_numpy(k).permute(1, 0, 2)[None]
    tv = torch.from_numpy(v).permute(1, 0, 2)[None]
    ref = F.scaled_dot_product_attention(tq, tk, tv, is_causal=True,
                                         enable_gqa=(Hq != Hkv))[0].permute(1, 0, 2).numpy()
    np.testing.assert_allclose(om.causal_attention(q, np.arange(T), k, v), ref,
                               rtol=1e-10, atol=1e-12)


def test_bf16_round_as_keeps_the_type():
    """bf16 rounding of float32 values stays float32 and equals torch's
    float32 -> bf16 conversion; of float64 values it equals bf16_round."""
    x = RNG.standard_normal(50000).astype(np.float32) * np.float32(5.0)
    got = on.bf16_round_as(x)
    assert got.dtype == np.float32
    np.testing.assert_array_equal(got, torch.from_numpy(x).to(torch.bfloat16).float().numpy())
    y = RNG.standard_normal(1000)
    got64 = on.bf16_round_as(y)
    assert got64.dtype == np.float64
    np.testing.assert_array_equal(got64, on.bf16_round(y))
