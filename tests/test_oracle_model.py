"""Pins for the oracle's model f (Preliminaries): each layer op against an independent library
routine or a closed form, the whole forward against an independent implementation of the same
architecture (Hugging Face ``LlamaForCausalLM``: pre-norm RMSNorm, rotate-half RoPE, GQA,
SwiGLU, tied embeddings), and the cached incremental forward against full recomputation."""
import numpy as np
import pytest
import torch

from oracle import model as om
from paper_2609_36590_amd import synth

TINY_GQA = synth.Config("t-gqa", 3, 1, 64, 4, 2, 16, 96, 101, 1e4, dtype=synth.F32)
TINY_MHA = synth.Config("t-mha", 2, 1, 48, 3, 3, 16, 80, 67, 5e3, dtype=synth.F32)


def _model(cfg, seed=0, dtype=np.float64, std=0.02):
    return om.Model(cfg, synth.make_weights(cfg, seed=seed, std=std), dtype=dtype)


def test_rmsnorm_matches_torch():
    rng = np.random.default_rng(0)
    x = rng.standard_normal((5, 33))
    g = rng.standard_normal(33)
    ref = torch.nn.functional.rms_norm(torch.from_numpy(x), (33,), torch.from_numpy(g), eps=1e-6)
    np.testing.assert_allclose(om.rmsnorm(x, g, 1e-6), ref.numpy(), rtol=1e-13, atol=1e-13)


def test_silu_matches_torch():
    x = np.linspace(-20, 20, 401)
    np.testing.assert_allclose(om.silu(x), torch.nn.functional.silu(torch.from_numpy(x)).numpy(),
                               rtol=1e-13, atol=1e-15)


def test_rope_is_complex_rotation():
    # Closed form: (x_i + i x_{i+d/2}) * exp(i * pos * base^(-2i/d)).
    rng = np.random.default_rng(1)
    d, base = 16, 1e4
    x = rng.standard_normal((7, 3, d))
    pos = np.array([0, 1, 2, 5, 100, 1000, 17000])
    cos, sin = om.rope_cos_sin(pos, d, base)
    y = om.apply_rope(x, cos, sin)
    z = x[..., :d // 2] + 1j * x[..., d // 2:]
    theta = base ** (-np.arange(d // 2) * 2.0 / d)
    rot = z * np.exp(1j * pos[:, None, None] * theta[None, None, :])
    np.testing.assert_allclose(y[..., :d // 2], rot.real, atol=1e-12)
    np.testing.assert_allclose(y[..., d // 2:], rot.imag, atol=1e-12)
    # position 0 is the identity, and rotations preserve norms
    np.testing.assert_allclose(y[0], x[0], atol=0)
    np.testing.assert_allclose(np.linalg.norm(y, axis=-1), np.linalg.norm(x, axis=-1), rtol=1e-12)


def test_rope_scores_depend_on_relative_position_only():
    rng = np.random.default_rng(2)
    d = 32
    q = rng.standard_normal((1, 1, d))
    k = rng.standard_normal((1, 1, d))

    def score(m, n):
        cq, sq = om.rope_cos_sin([m], d, 1e6)
        ck, sk = om.rope_cos_sin([n], d, 1e6)
        return float(np.sum(om.apply_rope(q, cq, sq) * om.apply_rope(k, ck, sk)))

    assert abs(score(10, 3) - score(110, 103)) < 1e-10
    assert abs(score(10, 3) - score(10, 4)) > 1e-6


@pytest.mark.parametrize("nh,nkv", [(4, 4), (8, 2), (6, 1)])
def test_attention_matches_torch_sdpa(nh, nkv):
    rng = np.random.default_rng(3)
    L, R, d = 23, 5, 16
    p = L - R
    q = rng.standard_normal((R, nh, d))
    K = rng.standard_normal((L, nkv, d))
    V = rng.standard_normal((L, nkv, d))
    pos = np.arange(p, p + R)
    ours = om.attention(q, K, V, pos)
    mask = torch.from_numpy(np.arange(L)[None, :] <= pos[:, None])
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q.transpose(1, 0, 2))[None], torch.from_numpy(K.transpose(1, 0, 2))[None],
        torch.from_numpy(V.transpose(1, 0, 2))[None], attn_mask=mask, enable_gqa=True)
    np.testing.assert_allclose(ours, ref[0].numpy().transpose(1, 0, 2), rtol=1e-11, atol=1e-12)


def test_attention_single_position_returns_value():
    rng = np.random.default_rng(4)
    q = rng.standard_normal((1, 2, 8))
    K = rng.standard_normal((1, 1, 8))
    V = rng.standard_normal((1, 1, 8))
    np.testing.assert_allclose(om.attention(q, K, V, [0]), np.repeat(V, 2, axis=1), atol=0)


def _hf_llama(cfg, weights):
    from transformers import LlamaConfig, LlamaForCausalLM

    hc = LlamaConfig(vocab_size=cfg.vocab, hidden_size=cfg.hidden, intermediate_size=cfg.ffn,
                     num_hidden_layers=cfg.n_layers, num_attention_heads=cfg.n_heads,
                     num_key_value_heads=cfg.n_kv_heads, head_dim=cfg.head_dim,
                     rms_norm_eps=cfg.rms_eps, rope_theta=cfg.rope_base,
                     tie_word_embeddings=True, attention_bias=False, mlp_bias=False,
                     max_position_embeddings=4096)
    m = LlamaForCausalLM(hc).double().eval()
    sd = {"model.embed_tokens.weight": weights["embed"], "model.norm.weight": weights["final_norm"],
          "lm_head.weight": weights["embed"]}
    names = {"wq": "self_attn.q_proj", "wk": "self_attn.k_proj", "wv": "self_attn.v_proj",
             "wo": "self_attn.o_proj", "w_gate": "mlp.gate_proj", "w_up": "mlp.up_proj",
             "w_down": "mlp.down_proj", "attn_norm": "input_layernorm",
             "mlp_norm": "post_attention_layernorm"}
    for i in range(cfg.n_layers):
        for ours, theirs in names.items():
            sd[f"model.layers.{i}.{theirs}.weight"] = weights[f"layers.{i}.{ours}"]
    m.load_state_dict({k: torch.from_numpy(np.asarray(v, dtype=np.float64)) for k, v in sd.items()},
                      strict=False)
    return m


@pytest.mark.parametrize("cfg", [TINY_GQA, TINY_MHA, synth.C1_TINY], ids=lambda c: c.name)
def test_full_forward_matches_hf_llama(cfg):
    # std 0.2 makes attention far from uniform so that a wrong mask, scale or rotation shows up.
    w = synth.make_weights(cfg, seed=5, std=0.2 if cfg.hidden < 200 else 0.05)
    tokens = np.random.default_rng(6).integers(0, cfg.vocab, size=40)
    ours = om.full_forward(om.Model(cfg, w, np.float64), tokens)
    with torch.no_grad():
        ref = _hf_llama(cfg, w)(torch.from_numpy(tokens)[None]).logits[0].numpy()
    scale = np.abs(ref).max()
    # the library forms its rotary angles in float32; positions < 40 keep that below 1e-5.
    assert np.abs(ours - ref).max() <= 2e-5 * max(1.0, scale), np.abs(ours - ref).max()


def test_cached_incremental_equals_full_recompute():
    cfg = TINY_GQA
    m = _model(cfg, std=0.2)
    toks = np.random.default_rng(7).integers(0, cfg.vocab, size=30)
    full = om.full_forward(m, toks)
    cache = om.KVCache(cfg, 64, np.float64)
    out = om.run_layers(m, cache, range(cfg.n_layers), m.embed(toks[:11]), 0)
    np.testing.assert_allclose(m.head(out), full[:11], rtol=1e-10, atol=1e-12)
    for s in range(11, 30):
        h = om.run_layers(m, cache, range(cfg.n_layers), m.embed(toks[s:s + 1]), s)
        np.testing.assert_allclose(m.head(h)[0], full[s], rtol=1e-10, atol=1e-12)


def test_full_forward_row_blocks_do_not_change_results():
    cfg = TINY_MHA
    m = _model(cfg, std=0.2)
    toks = np.random.default_rng(8).integers(0, cfg.vocab, size=37)
    np.testing.assert_allclose(om.full_forward(m, toks, row_block=5),
                               om.full_forward(m, toks, row_block=256), rtol=1e-12, atol=1e-13)


def test_kvcache_rejects_gaps_and_reads_past_valid():
    cfg = TINY_MHA
    c = om.KVCache(cfg, 8, np.float64)
    k = np.zeros((2, cfg.n_kv_heads, cfg.head_dim))
    c.append(0, 0, k, k)
    with pytest.raises(AssertionError):
        c.append(0, 3, k, k)
    with pytest.raises(AssertionError):
        c.prefix(0, 3)
    c.truncate(1)
    assert c.valid[0] == 1


def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(9)
    x = np.concatenate([rng.standard_normal(4000) * 10.0 ** rng.integers(-8, 8, 4000),
                        [0.0, -0.0, 1.0, 1.00390625, 1.01171875, 65504.0, 3.0e38]])
    ref = torch.from_numpy(x.astype(np.float32)).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(om.round_to_bf16(x), ref)


def test_bf16_model_rounds_kv_only():
    cfg = TINY_GQA.replace(dtype=synth.BF16)
    w = synth.weights_as_f32(cfg, synth.make_weights(cfg, seed=1, std=0.2))
    toks = np.random.default_rng(3).integers(0, cfg.vocab, size=12)
    exact = om.Model(cfg, w, np.float64, kv_bf16=False)
    rounded = om.Model(cfg, w, np.float64)
    assert rounded.kv_bf16 and not exact.kv_bf16
    _, K, V = om.full_forward(rounded, toks, return_kv=True)
    np.testing.assert_array_equal(om.round_to_bf16(K), K)
    np.testing.assert_array_equal(om.round_to_bf16(V), V)
    d = np.abs(om.full_forward(rounded, toks) - om.full_forward(exact, toks)).max()
    assert 0 < d < 0.2  # bf16 storage is a small but visible perturbation


def test_sampled_first_layer_kv_match_hf_llama_cache():
    # Layer 0 and 1 keys/values formed one position at a time (the route the full-size GPU tests
    # take at 16k tokens) against the key/value cache of the independent implementation.
    cfg = TINY_GQA
    w = synth.make_weights(cfg, seed=5, std=0.2)
    tokens = np.random.default_rng(6).integers(0, cfg.vocab, size=40)
    pos = [0, 1, 16, 17, 39]
    got = om.sampled_kv_first_layers(om.Model(cfg, w, np.float64), tokens, pos)
    with torch.no_grad():
        pkv = _hf_llama(cfg, w)(torch.from_numpy(tokens)[None], use_cache=True).past_key_values
    for layer in (0, 1):
        for j, name in ((0, "keys"), (1, "values")):
            t = getattr(pkv.layers[layer], name)                     # [1, n_kv, seq, d]
            ref = t[0].numpy().transpose(1, 0, 2)[pos]                  # [n, n_kv, d]
            ours = got[2 * layer + j]
            err = np.abs(ours - ref).max()
            assert err <= 2e-5 * max(1.0, np.abs(ref).max()), (layer, name, err)


def test_layer_kv_equals_block_keys_values():
    cfg = TINY_MHA.replace(dtype=synth.BF16)
    w = synth.weights_as_f32(cfg, synth.make_weights(cfg, seed=2, std=0.2))
    m = om.Model(cfg, w, np.float64)
    h = m.embed(np.random.default_rng(4).integers(0, cfg.vocab, size=6))
    empty = np.zeros((3, cfg.n_kv_heads, cfg.head_dim))
    _, k, v = m.block(1, h, np.arange(3, 9), empty, empty)
    k2, v2 = m.kv(1, h, np.arange(3, 9))
    np.testing.assert_array_equal(k2, k)
    np.testing.assert_array_equal(v2, v)
