"""The oracle's pins catch plausible mistakes.

Each case plants one mistake in a copy of an oracle function (by editing its
source text), installs it with monkeypatch, and checks that at least one pin
(the transformers comparison, brute-force attention, the decode identity)
now fails.  Mistakes live only in the oracle and only on the CPU."""
import inspect
import textwrap

import numpy as np
import pytest

from oracle import model as om
import test_oracle_model as tm
import test_oracle_ops as to

MUTATIONS = [
    ("rope", "x1 * c - x2 * s, x2 * c + x1 * s", "x1 * c + x2 * s, x2 * c - x1 * s"),
    ("rope", "(2.0 * np.arange(half, dtype=np.float64)) / d", "(np.arange(half, dtype=np.float64)) / d"),
    ("causal_attention", "kh = h // G", "kh = h % Hkv"),
    ("causal_attention", "key_pos[None, :] <= np.asarray(q_pos)[:, None]",
     "key_pos[None, :] < np.asarray(q_pos)[:, None] + (np.asarray(q_pos)[:, None] == 0)"),
    ("causal_attention", "scale = 1.0 / math.sqrt(d)", "scale = 1.0"),
    ("rmsnorm", "x / np.sqrt(ms + eps) * g", "x / np.sqrt(ms + eps)"),
    ("layer", "a = rnd(silu(gu[:, :F]) * gu[:, F:])", "a = rnd(silu(gu[:, F:]) * gu[:, :F])"),
    ("layer", "r = r + o @ f64(w[\"w_o\"]).T", "r = o @ f64(w[\"w_o\"]).T"),
    ("layer", "h2 = rnd(rmsnorm(r, f64(w[\"mlp_norm\"]), shp.rms_eps))",
     "h2 = rnd(rmsnorm(r, f64(w[\"attn_norm\"]), shp.rms_eps))"),
    ("qkv_heads", "q = rnd(rope(q, pos, shp.rope_theta))", "q = rnd(q)"),
    ("qkv_heads", "k = qkv[:, Hq * d:(Hq + Hkv) * d].reshape(T, Hkv, d)",
     "k = qkv[:, Hq * d:(Hq + Hkv) * d].reshape(T, d, Hkv).transpose(0, 2, 1)"),
    ("decode", "K_cache[l][:n], V_cache[l][:n]", "K_cache[l][:n - 1], V_cache[l][:n - 1]"),
    ("decode", "pos = np.array([n])", "pos = np.array([n - 1])"),
    ("prefill_chunk", "pos = start + np.arange(len(ids))", "pos = np.arange(len(ids))"),
    ("prefill_chunk", "kp = K_cache[l][:start] if start > 0 else None",
     "kp = K_cache[l][:start - 1] if start > 1 else None"),
]


def mutated(name, old, new):
    src = textwrap.dedent(inspect.getsource(getattr(om, name)))
    assert old in src, (name, old)
    ns = dict(om.__dict__)
    exec(compile(src.replace(old, new), f"<mutant {name}>", "exec"), ns)
    return ns[name]


def pins():
    yield lambda: tm.test_unrounded_forward_matches_transformers(True)
    yield lambda: tm.test_unrounded_forward_matches_transformers(False)
    yield to.test_attention_brute_force_gqa
    yield to.test_attention_decode_row_brute_force
    yield lambda: to.test_attention_matches_torch_sdpa(8, 2)
    yield to.test_rope_matches_complex_rotation
    yield to.test_rmsnorm_matches_torch
    yield lambda: tm.test_decode_equals_last_prefill_row(True)
    yield lambda: tm.test_chunked_prefill_equals_whole_prefill(False)


@pytest.mark.parametrize("name,old,new", MUTATIONS, ids=[f"{m[0]}-{i}" for i, m in enumerate(MUTATIONS)])
def test_pins_catch_mutation(monkeypatch, name, old, new):
    monkeypatch.setattr(om, name, mutated(name, old, new))
    caught = 0
    for pin in pins():
        try:
            pin()
        except (AssertionError, ValueError, IndexError):
            caught += 1
            break
    assert caught, f"no pin caught the mutation in {name}: {new}"
