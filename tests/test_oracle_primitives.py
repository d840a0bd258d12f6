"""Pins for the oracle's building blocks (CPU only).

Each test ties an oracle function to something other than itself: a torch.nn.functional routine,
an independent formulation (complex rotation), a closed form, or an invariant."""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

import synth
from oracle import model as om

RNG = np.random.default_rng(1234)


def test_rms_norm_matches_torch_routine():
    x = RNG.standard_normal((5, 96))
    g = RNG.standard_normal(96)
    ref = F.rms_norm(torch.from_numpy(x), (96,), torch.from_numpy(g), eps=1e-6).numpy()
    np.testing.assert_allclose(om.rms_norm(x, g, 1e-6), ref, rtol=1e-12, atol=1e-12)


def test_rms_norm_closed_forms():
    # constant vector c*1 with unit gain maps to c / sqrt(c^2 + eps)
    c, eps = 0.37, 1e-6
    y = om.rms_norm(np.full(64, c), np.ones(64), eps)
    np.testing.assert_allclose(y, c / np.sqrt(c * c + eps), rtol=1e-14)
    # unit gain, eps=0: root mean square of the output is exactly 1; scale invariant
    x = RNG.standard_normal(128)
    y = om.rms_norm(x, np.ones(128), 0.0)
    assert abs(np.sqrt(np.mean(y * y)) - 1) < 1e-14
    np.testing.assert_allclose(om.rms_norm(7.5 * x, np.ones(128), 0.0), y, rtol=1e-13)
    # the zero vector stays zero (eps keeps it finite)
    assert np.all(om.rms_norm(np.zeros(8), np.ones(8), 1e-6) == 0)


def test_silu_matches_torch_routine():
    x = RNG.standard_normal(1000) * 5
    np.testing.assert_allclose(om.silu(x), F.silu(torch.from_numpy(x)).numpy(), rtol=1e-13, atol=1e-15)


def test_rope_equals_complex_rotation():
    # channel j and j+dh/2 as the complex number x_j + i x_{j+dh/2}, multiplied by e^{i p theta_j}
    dh, base = 64, 10000.0
    x = RNG.standard_normal((3, dh))
    for p in [0, 1, 17, 1000, 32767]:
        z = x[:, : dh // 2] + 1j * x[:, dh // 2:]
        theta = base ** (-np.arange(0, dh, 2) / dh)
        zr = z * np.exp(1j * p * theta)
        ref = np.concatenate([zr.real, zr.imag], axis=-1)
        np.testing.assert_allclose(om.rope(x, p, base), ref, rtol=1e-12, atol=1e-12)


def test_rope_invariants():
    dh, base = 128, 10000.0
    q = RNG.standard_normal((1, dh))
    k = RNG.standard_normal((1, dh))
    assert np.array_equal(om.rope(q, 0, base), q)  # position 0 is the identity
    for p in [3, 250, 9000]:
        assert abs(np.linalg.norm(om.rope(q, p, base)) - np.linalg.norm(q)) < 1e-12
    # <R_p q, R_p' k> depends only on p - p'
    d1 = float((om.rope(q, 40, base) @ om.rope(k, 30, base).T)[0, 0])
    d2 = float((om.rope(q, 1010, base) @ om.rope(k, 1000, base).T)[0, 0])
    assert abs(d1 - d2) < 1e-10


def test_attend_matches_torch_sdpa_gqa():
    hq, hkv, dh, T = 8, 2, 32, 37
    q = RNG.standard_normal((hq, dh))
    cache = om.LayerCache(hkv, dh, 4)
    for t in range(T):
        cache.append(t, RNG.standard_normal((hkv, dh)), RNG.standard_normal((hkv, dh)))
    upto = 29
    o = om.attend(q, cache, upto)
    Q = torch.from_numpy(q)[None, :, None, :]  # [1, Hq, 1, dh]
    K = torch.from_numpy(cache.k[: upto + 1]).permute(1, 0, 2)[None]  # [1, Hkv, T, dh]
    V = torch.from_numpy(cache.v[: upto + 1]).permute(1, 0, 2)[None]
    ref = F.scaled_dot_product_attention(Q, K, V, enable_gqa=True)[0, :, 0, :].reshape(-1).numpy()
    np.testing.assert_allclose(o, ref, rtol=1e-12, atol=1e-12)


def test_attend_closed_forms():
    hq, hkv, dh = 4, 2, 16
    cache = om.LayerCache(hkv, dh, 4)
    k = RNG.standard_normal((hkv, dh))
    vs = []
    for t in range(6):  # identical keys -> uniform weights -> output is the mean of the values
        v = RNG.standard_normal((hkv, dh))
        vs.append(v)
        cache.append(t, k, v)
    q = RNG.standard_normal((hq, dh))
    o = om.attend(q, cache, 5).reshape(hq, dh)
    mean_v = np.mean(vs, axis=0)
    for h in range(hq):
        np.testing.assert_allclose(o[h], mean_v[h // 2], rtol=1e-12)
    # one key: the output is that key's value
    o1 = om.attend(q, cache, 0).reshape(hq, dh)
    for h in range(hq):
        np.testing.assert_allclose(o1[h], vs[0][h // 2], rtol=1e-14)


def test_argmax_lowest_index_on_ties():
    v = np.array([0.1, 0.5, -1.0, 0.5, 0.5])
    assert om.argmax_first(v) == 1
    assert om.argmax_first(np.zeros(10)) == 0


def test_round_bf16_matches_storage_rounding():
    # the oracle's float64 -> bf16 rounding agrees with the input generator's fp32 -> bf16 rounding
    x = (RNG.standard_normal(100000) * np.exp(RNG.uniform(-20, 20, 100000))).astype(np.float32)
    ref = synth.bf16_bits_to_f32(synth.bf16_bits(x)).astype(np.float64)
    np.testing.assert_array_equal(om.round_bf16(x.astype(np.float64)), ref)
    # ties go to even: 1 + 2^-8 lies halfway between 1 and 1 + 2^-7
    assert om.round_bf16(np.array([1 + 2.0 ** -8]))[0] == 1.0
    assert om.round_bf16(np.array([1 + 3 * 2.0 ** -8]))[0] == 1 + 2.0 ** -6


def _hf_llama(shape, model):
    from transformers import LlamaConfig, LlamaForCausalLM
    cfg = LlamaConfig(vocab_size=shape.vocab, hidden_size=shape.d_model, intermediate_size=shape.ffn_dim,
                      num_hidden_layers=shape.n_layers, num_attention_heads=shape.n_q_heads,
                      num_key_value_heads=shape.n_kv_heads, head_dim=shape.head_dim,
                      rms_norm_eps=shape.rms_eps, rope_theta=shape.rope_base, tie_word_embeddings=False,
                      attention_bias=False, mlp_bias=False, max_position_embeddings=4096)
    cfg._attn_implementation = "eager"
    hf = LlamaForCausalLM(cfg).double().eval()
    sd = {"model.embed_tokens.weight": model.w("embed"), "model.norm.weight": model.w("final_norm"),
          "lm_head.weight": model.w("lm_head")}
    names = {"wq": "self_attn.q_proj", "wk": "self_attn.k_proj", "wv": "self_attn.v_proj",
             "wo": "self_attn.o_proj", "wg": "mlp.gate_proj", "wu": "mlp.up_proj", "wd": "mlp.down_proj",
             "attn_norm": "input_layernorm", "mlp_norm": "post_attention_layernorm"}
    for l in range(shape.n_layers):
        for k, v in names.items():
            sd[f"model.layers.{l}.{v}.weight"] = model.w(f"layer.{l}.{k}")
    hf.load_state_dict({k: torch.from_numpy(np.ascontiguousarray(v)) for k, v in sd.items()}, strict=True)
    return hf


def test_target_model_matches_transformers_llama():
    """The oracle's decoder (cached, one position at a time) against the transformers Llama
    implementation of the same architecture, on the tiny workload's weights."""
    sh = synth.TINY
    model = om.Model(sh, seed=3)
    prompt = synth.prompt(sh, 3, 40)
    hf = _hf_llama(sh, model)
    with torch.no_grad():
        out = hf(torch.from_numpy(prompt.astype(np.int64))[None], output_hidden_states=True)
    ref_logits = out.logits[0].numpy()
    caches = om.new_caches(sh, sh.n_layers)
    for p, t in enumerate(prompt):
        h, kept = om.run_token(model, caches, int(t), p, keep=list(range(sh.n_layers)))
        for l in range(sh.n_layers):  # hidden_states[l] is H^l for l < L
            np.testing.assert_allclose(kept[l], out.hidden_states[l][0, p].numpy(), rtol=1e-5, atol=1e-6)
        lg = om.lm_logits(model, h)
        np.testing.assert_allclose(lg, ref_logits[p], rtol=1e-5, atol=1e-6)
    # and the no-cache brute force agrees with the cached path at every layer
    full = om.forward_full(model, prompt)
    np.testing.assert_allclose(om.lm_logits(model, full[sh.n_layers][-1]), ref_logits[-1], rtol=1e-5, atol=1e-6)
