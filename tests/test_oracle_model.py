"""Oracle pins for the whole decoder forward.

* Library special case: with rounding switched off the oracle's K/V cache and
  logits equal those of an independent implementation of the same model
  families (transformers' Qwen3 with QK-norm, Llama without), run in float64.
* Causality: the K/V of a prefix prefill equal the first rows of a prefill
  over the whole context (the stable-prefix premise of Sections 3 and 4.3).
* KV-cache identity: a decode step at position n over the cache of [0, n)
  gives the logits of the last row of a prefill over n + 1 tokens
  (decoding resumes at n without re-running prefill, Section 4.3).
"""
import numpy as np
import pytest
import torch

from oracle import model as om
from oracle import numerics as on
from workloads import configs, gen
from helpers import oracle_weights, shape_of

transformers = pytest.importorskip("transformers")


def small_cfg(qk_norm, **kw):
    base = dict(name="t", n_layers=2, hidden=64, n_q_heads=4, n_kv_heads=2,
                head_dim=32, ffn=96, vocab=128, qk_norm=qk_norm, rope_theta=1e4)
    base.update(kw)
    return configs.ModelConfig(**base)


def hf_model(cfg, glob, layers):
    if cfg.qk_norm:
        from transformers import Qwen3Config, Qwen3ForCausalLM
        hc = Qwen3Config(vocab_size=cfg.vocab, hidden_size=cfg.hidden,
                         intermediate_size=cfg.ffn, num_hidden_layers=cfg.n_layers,
                         num_attention_heads=cfg.n_q_heads, num_key_value_heads=cfg.n_kv_heads,
                         head_dim=cfg.head_dim, rms_norm_eps=cfg.rms_eps,
                         rope_theta=cfg.rope_theta, tie_word_embeddings=False,
                         attention_bias=False, max_position_embeddings=4096)
        m = Qwen3ForCausalLM(hc)
    else:
        from transformers import LlamaConfig, LlamaForCausalLM
        hc = LlamaConfig(vocab_size=cfg.vocab, hidden_size=cfg.hidden,
                         intermediate_size=cfg.ffn, num_hidden_layers=cfg.n_layers,
                         num_attention_heads=cfg.n_q_heads, num_key_value_heads=cfg.n_kv_heads,
                         head_dim=cfg.head_dim, rms_norm_eps=cfg.rms_eps,
                         rope_theta=cfg.rope_theta, tie_word_embeddings=False,
                         attention_bias=False, mlp_bias=False, max_position_embeddings=4096)
        m = LlamaForCausalLM(hc)
    hc._attn_implementation = "eager"
    m = m.to(torch.float64).eval()
    qd, kd = cfg.q_dim, cfg.kv_dim
    F = cfg.ffn
    with torch.no_grad():
        m.model.embed_tokens.weight.copy_(glob["embed"].double())
        m.model.norm.weight.copy_(glob["final_norm"].double())
        m.lm_head.weight.copy_(glob["lm_head"].double())
        for l, w in enumerate(layers):
            L = m.model.layers[l]
            qkv = w["w_qkv"].double()
            L.self_attn.q_proj.weight.copy_(qkv[:qd])
            L.self_attn.k_proj.weight.copy_(qkv[qd:qd + kd])
            L.self_attn.v_proj.weight.copy_(qkv[qd + kd:])
            L.self_attn.o_proj.weight.copy_(w["w_o"].double())
            if cfg.qk_norm:
                L.self_attn.q_norm.weight.copy_(w["q_norm"].double())
                L.self_attn.k_norm.weight.copy_(w["k_norm"].double())
            L.input_layernorm.weight.copy_(w["attn_norm"].double())
            L.post_attention_layernorm.weight.copy_(w["mlp_norm"].double())
            gu = w["w_gate_up"].double()
            L.mlp.gate_proj.weight.copy_(gu[:F])
            L.mlp.up_proj.weight.copy_(gu[F:])
            L.mlp.down_proj.weight.copy_(w["w_down"].double())
    return m


def hf_kv_and_logits(m, ids):
    with torch.no_grad():
        out = m(torch.tensor([ids]), use_cache=True)
    pkv = out.past_key_values
    K, V = [], []
    for l in range(len(m.model.layers)):
        if hasattr(pkv, "layers"):
            k, v = pkv.layers[l].keys, pkv.layers[l].values
        else:
            k, v = pkv[l]
        K.append(k[0].permute(1, 0, 2).numpy())
        V.append(v[0].permute(1, 0, 2).numpy())
    return K, V, out.logits[0].numpy()


@pytest.mark.parametrize("qk_norm", [True, False])
def test_unrounded_forward_matches_transformers(qk_norm):
    cfg = small_cfg(qk_norm)
    glob, layers = gen.model_weights(cfg, seed=3, gain_sigma=0.1)
    # larger weights so every term matters at the comparison tolerance
    glob = {k: (v.float() * (5.0 if v.dim() == 2 else 1.0)).to(torch.bfloat16) for k, v in glob.items()}
    layers = [{k: (v.float() * (5.0 if v.dim() == 2 else 1.0)).to(torch.bfloat16)
               for k, v in l.items()} for l in layers]
    ids = gen.token_ids(19, cfg.vocab, seed=3).tolist()
    m = hf_model(cfg, glob, layers)
    Kr, Vr, logit_r = hf_kv_and_logits(m, ids)
    g, ls = oracle_weights(glob, layers)
    shp = shape_of(cfg)
    K, V, r = om.prefill(ids, g, ls, shp, rnd=on.no_round, full_last=True)
    lg = om.logits(r, g, shp, rnd=on.no_round)
    # transformers evaluates RMSNorm and the rotary angles in float32
    for l in range(cfg.n_layers):
        for a, b in ((K[l], Kr[l]), (V[l], Vr[l])):
            assert np.max(np.abs(a - b)) <= 2e-5 * np.max(np.abs(b))
    assert np.max(np.abs(lg - logit_r)) <= 2e-5 * np.max(np.abs(logit_r))


def test_causality_prefix_equals_full_rows():
    cfg = configs.TINY
    glob, layers = gen.model_weights(cfg, seed=0)
    g, ls = oracle_weights(glob, layers)
    shp = shape_of(cfg)
    ids = gen.token_ids(128, cfg.vocab, seed=0).tolist()
    Kf, Vf, _ = om.prefill(ids, g, ls, shp)
    Kp, Vp, _ = om.prefill(ids[:96], g, ls, shp)
    for l in range(cfg.n_layers):
        # same rows, same arithmetic: equal up to float64 summation order
        # (bf16 rounding could only flip on an exact float64 tie)
        np.testing.assert_allclose(Kp[l], Kf[l][:96], rtol=1e-9, atol=1e-12)
        np.testing.assert_allclose(Vp[l], Vf[l][:96], rtol=1e-9, atol=1e-12)


@pytest.mark.parametrize("qk_norm", [False, True])
def test_chunked_prefill_equals_whole_prefill(qk_norm):
    """A prefix prefilled chunk by chunk (ragged chunks, starts not
    multiples of 16 or 32) gives the K/V of one prefill over the whole
    prefix: each chunk's tokens see the earlier chunks through the cache."""
    cfg = configs.TINY.replace(qk_norm=qk_norm)
    glob, layers = gen.model_weights(cfg, seed=4, gain_sigma=0.1)
    g, ls = oracle_weights(glob, layers)
    shp = shape_of(cfg)
    ids = gen.token_ids(100, cfg.vocab, seed=4).tolist()
    Kf, Vf, _ = om.prefill(ids, g, ls, shp)
    K = [np.zeros((0,) + k.shape[1:]) for k in Kf]
    V = [np.zeros((0,) + v.shape[1:]) for v in Vf]
    for a, b in ((0, 37), (37, 38), (38, 80), (80, 100)):
        kc, vc = om.prefill_chunk(ids[a:b], a, K, V, g, ls, shp)
        K = [np.concatenate([K[l], kc[l]]) for l in range(cfg.n_layers)]
        V = [np.concatenate([V[l], vc[l]]) for l in range(cfg.n_layers)]
    for l in range(cfg.n_layers):
        np.testing.assert_allclose(K[l], Kf[l], rtol=1e-9, atol=1e-12)
        np.testing.assert_allclose(V[l], Vf[l], rtol=1e-9, atol=1e-12)


@pytest.mark.parametrize("qk_norm", [False, True])
def test_decode_equals_last_prefill_row(qk_norm):
    cfg = configs.TINY.replace(qk_norm=qk_norm)
    glob, layers = gen.model_weights(cfg, seed=1, gain_sigma=0.1)
    g, ls = oracle_weights(glob, layers)
    shp = shape_of(cfg)
    ids = gen.token_ids(41, cfg.vocab, seed=1).tolist()
    n = 40
    K, V, _ = om.prefill(ids[:n], g, ls, shp)
    lg, kn, vn = om.decode(ids[n], n, K, V, g, ls, shp)
    Kf, Vf, rf = om.prefill(ids, g, ls, shp, full_last=True)
    ref = om.logits(rf[-1:], g, shp)[0]
    np.testing.assert_allclose(lg, ref, rtol=1e-9, atol=1e-9 * np.max(np.abs(ref)))
    for l in range(cfg.n_layers):
        np.testing.assert_allclose(kn[l][0], Kf[l][n], rtol=1e-9, atol=1e-12)
        np.testing.assert_allclose(vn[l][0], Vf[l][n], rtol=1e-9, atol=1e-12)


def test_bf16_rounding_drift_is_small():
    """The rounded forward stays within the parity tolerance of the exact one
    at the tiny shape: the rounding points do not dominate the values."""
    cfg = configs.TINY
    glob, layers = gen.model_weights(cfg, seed=2)
    g, ls = oracle_weights(glob, layers)
    shp = shape_of(cfg)
    ids = gen.token_ids(64, cfg.vocab, seed=2).tolist()
    K1, V1, _ = om.prefill(ids, g, ls, shp)
    K0, V0, _ = om.prefill(ids, g, ls, shp, rnd=on.no_round)
    for l in range(cfg.n_layers):
        assert np.max(np.abs(K1[l] - K0[l])) <= 1e-2 * np.max(np.abs(K0[l]))
        assert np.max(np.abs(V1[l] - V0[l])) <= 1e-2 * np.max(np.abs(V0[l]))


def test_precision_float32_evaluation():
    """``precision(np.float32)`` evaluates the same forward in float32 and
    restores float64 on exit.  Pinned against the float64 forward (itself
    pinned to transformers above): unrounded, the float32 cache and logits
    agree within float32 accuracy, every result is float32 inside the
    context and float64 after it; and with bf16 rounding at the stored
    points (``bf16_round_as``) the float32 cache holds bf16 values."""
    cfg = small_cfg(True)
    glob, layers = gen.model_weights(cfg, seed=5, gain_sigma=0.1)
    ids = gen.token_ids(23, cfg.vocab, seed=5).tolist()
    g, ls = oracle_weights(glob, layers)
    shp = shape_of(cfg)
    K, V, r = om.prefill(ids, g, ls, shp, rnd=on.no_round, full_last=True)
    lg = om.logits(r, g, shp, rnd=on.no_round)
    keep = lambda x: x   # noqa: E731  (no rounding, type kept)
    with om.precision(np.float32):
        g32 = {k: v.astype(np.float32) for k, v in g.items()}
        ls32 = [{k: v.astype(np.float32) for k, v in w.items()} for w in ls]
        K32, V32, r32 = om.prefill(ids, g32, ls32, shp, rnd=keep, full_last=True)
        lg32 = om.logits(r32, g32, shp, rnd=keep)
        Kb, _, _ = om.prefill(ids, g32, ls32, shp, rnd=on.bf16_round_as)
    for a in K32 + V32 + [r32, lg32] + Kb:
        assert a.dtype == np.float32
    for a, b in zip(K32 + V32 + [lg32], K + V + [lg]):
        assert 0 < np.max(np.abs(a - b)) <= 1e-5 * np.max(np.abs(b))
    for k in Kb:
        np.testing.assert_array_equal(k, torch.from_numpy(k).to(torch.bfloat16).float().numpy())
    K2, _, _ = om.prefill(ids, g, ls, shp, rnd=on.no_round)
    assert K2[0].dtype == np.float64
    np.testing.assert_array_equal(K2[0], K[0])
