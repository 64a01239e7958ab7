"""Pins for the oracle decoder forward pass (CPU)."""
import numpy as np
import pytest
import torch

import jf_inputs
from oracle.model import DecoderOracle
from oracle.numerics import round_bf16

SMALL = dict(n_layers=2, d_model=64, n_heads=4, n_kv_heads=2, head_dim=16,
             d_ffn=96, vocab=97, rope_base=10000.0, rms_eps=1e-6, dtype="f32")


def hf_llama(shape, weights):
    """transformers' Llama (rotate-half RoPE, RMSNorm, SwiGLU, GQA) in float64."""
    from transformers import LlamaConfig, LlamaForCausalLM
    cfg = LlamaConfig(vocab_size=shape["vocab"], hidden_size=shape["d_model"],
                      intermediate_size=shape["d_ffn"], num_hidden_layers=shape["n_layers"],
                      num_attention_heads=shape["n_heads"], num_key_value_heads=shape["n_kv_heads"],
                      head_dim=shape["head_dim"], rms_norm_eps=shape["rms_eps"],
                      rope_theta=shape["rope_base"], tie_word_embeddings=False,
                      attention_bias=False, mlp_bias=False, max_position_embeddings=4096)
    m = LlamaForCausalLM(cfg).double().eval()
    sd = {"model.embed_tokens.weight": weights["embed"], "model.norm.weight": weights["final_norm"],
          "lm_head.weight": weights["lm_head"]}
    for l in range(shape["n_layers"]):
        p, q = f"layers.{l}.", f"model.layers.{l}."
        sd.update({q + "input_layernorm.weight": weights[p + "attn_norm"],
                   q + "self_attn.q_proj.weight": weights[p + "wq"],
                   q + "self_attn.k_proj.weight": weights[p + "wk"],
                   q + "self_attn.v_proj.weight": weights[p + "wv"],
                   q + "self_attn.o_proj.weight": weights[p + "wo"],
                   q + "post_attention_layernorm.weight": weights[p + "ffn_norm"],
                   q + "mlp.gate_proj.weight": weights[p + "w_gate"],
                   q + "mlp.up_proj.weight": weights[p + "w_up"],
                   q + "mlp.down_proj.weight": weights[p + "w_down"]})
    m.load_state_dict({k: torch.from_numpy(np.asarray(v, np.float64)) for k, v in sd.items()})
    return m


@pytest.mark.parametrize("shape", [SMALL, jf_inputs.MODEL_SHAPES["tiny"]], ids=["gqa", "tiny"])
def test_forward_matches_transformers_llama(shape):
    """The whole forward (embedding, gains, RoPE pairing, GQA grouping, SwiGLU,
    untied head) equals an independent, widely used implementation."""
    w = jf_inputs.model_weights(shape, seed=3)
    toks = jf_inputs.prompt(5, 40, shape["vocab"])
    with torch.no_grad():
        ref = hf_llama(shape, w)(torch.from_numpy(toks.astype(np.int64))[None]).logits[0].numpy()
    m = DecoderOracle(shape, w)
    R = len(toks)
    logits, _ = m.forward(toks, np.arange(R), np.tri(R, dtype=bool))
    # transformers runs RMSNorm and the RoPE frequencies in float32 even in a
    # float64 model, so agreement is at float32 level; a structural mistake
    # (wrong pairing, transposed weight, dropped gain) moves logits by ~0.1.
    np.testing.assert_allclose(logits, ref, rtol=0, atol=2e-6)


def test_cached_prefix_equals_full_sequence_bitwise():
    """KV-cache invariant: rows run against a committed cache produce exactly
    the logits of the same rows inside one full causal pass (row invariance)."""
    w = jf_inputs.model_weights(SMALL, seed=4)
    toks = jf_inputs.prompt(6, 30, SMALL["vocab"])
    full = DecoderOracle(SMALL, w)
    lf, _ = full.forward(toks, np.arange(30), np.tri(30, dtype=bool))
    inc = DecoderOracle(SMALL, w)
    inc.prefill(toks[:11], chunk=4)
    li, _ = inc.forward(toks[11:], 11 + np.arange(19), np.tri(19, dtype=bool))
    assert np.array_equal(li, lf[11:])
    # and the cache equals the one a single prefill builds
    one = DecoderOracle(SMALL, w)
    one.prefill(toks[:11])
    for l in range(SMALL["n_layers"]):
        assert np.array_equal(one.K[l], inc.K[l]) and np.array_equal(one.Vc[l], inc.Vc[l])


def test_attention_matches_torch_sdpa_with_tree_mask():
    shape = dict(SMALL, n_heads=6, n_kv_heads=2, head_dim=16)
    m = DecoderOracle(shape, {}, compute=np.float64)
    rng = np.random.default_rng(1)
    C, R, G, H, hd = 9, 7, 2, 6, 16
    m.K[0] = rng.standard_normal((C, G, hd))
    m.Vc[0] = rng.standard_normal((C, G, hd))
    q = rng.standard_normal((R, H, hd))
    k = rng.standard_normal((R, G, hd))
    v = rng.standard_normal((R, G, hd))
    vis = np.tri(R, dtype=bool)
    vis[4, 1:4] = False      # a branch hanging under row 0
    vis[5, 1:4] = False
    vis[6] = False; vis[6, [0, 6]] = True
    out = m.attention(0, q, k, v, vis)
    keys = np.concatenate([m.K[0], k]); vals = np.concatenate([m.Vc[0], v])
    mask = np.concatenate([np.ones((R, C), bool), vis], axis=1)
    kt = torch.from_numpy(keys).permute(1, 0, 2).repeat_interleave(H // G, dim=0)
    vt = torch.from_numpy(vals).permute(1, 0, 2).repeat_interleave(H // G, dim=0)
    qt = torch.from_numpy(q).permute(1, 0, 2)
    ref = torch.nn.functional.scaled_dot_product_attention(
        qt, kt, vt, attn_mask=torch.from_numpy(mask)[None]).permute(1, 0, 2).numpy()
    np.testing.assert_allclose(out, ref, atol=1e-12)
    # the vectorised form used for large shapes computes the same thing
    m.row_invariant = False
    np.testing.assert_allclose(m.attention(0, q, k, v, vis), ref, atol=1e-12)


def test_rope_relative_position_invariant():
    m = DecoderOracle(SMALL, {})
    rng = np.random.default_rng(2)
    q = rng.standard_normal((1, 1, 16)); k = rng.standard_normal((1, 1, 16))
    base = np.sum(m.rope(q, [7]) * m.rope(k, [3]))
    for t in (1, 50, 900):
        assert abs(np.sum(m.rope(q, [7 + t]) * m.rope(k, [3 + t])) - base) < 1e-9
    # position 0 is the identity, and the rotation keeps the norm
    np.testing.assert_array_equal(m.rope(q, [0]), q)
    assert abs(np.linalg.norm(m.rope(q, [123])) - np.linalg.norm(q)) < 1e-12
    # pairing is (i, i + hd/2): a vector living on dims (0, 8) stays there
    e = np.zeros((1, 1, 16)); e[0, 0, 0] = 1.0
    r = m.rope(e, [1])[0, 0]
    assert abs(r[0] - np.cos(1.0)) < 1e-15 and abs(r[8] - np.sin(1.0)) < 1e-15
    assert np.count_nonzero(r) == 2


def test_rmsnorm_closed_form():
    m = DecoderOracle(SMALL, {})
    h = np.full((1, 64), -3.0)
    gain = np.linspace(0.5, 1.5, 64)
    y = m.rmsnorm(h, gain)
    np.testing.assert_allclose(y[0], -gain / np.sqrt(1.0 + 1e-6 / 9.0), rtol=1e-15)


def test_bf16_mode_rounding_points():
    """bf16 model: cached K/V are bf16 values, the rest is unrounded, so the
    logits stay close to a run without the cache rounding."""
    shape = dict(SMALL, dtype="bf16")
    w = jf_inputs.model_weights(shape, seed=8)
    toks = jf_inputs.prompt(9, 12, shape["vocab"])
    m = DecoderOracle(shape, w)
    m.prefill(toks)
    for l in range(shape["n_layers"]):
        assert np.array_equal(round_bf16(m.K[l]), m.K[l])
        assert np.array_equal(round_bf16(m.Vc[l]), m.Vc[l])
    exact = DecoderOracle(shape, w)
    exact.bf16 = False
    lb, _ = m.forward(toks[:3], 12 + np.arange(3), np.tri(3, dtype=bool))
    exact.prefill(toks)
    le, _ = exact.forward(toks[:3], 12 + np.arange(3), np.tri(3, dtype=bool))
    assert 0 < np.abs(lb - le).max() < 0.05


def test_float32_batched_mode_close_to_fp64():
    w = jf_inputs.model_weights(SMALL, seed=10)
    toks = jf_inputs.prompt(11, 20, SMALL["vocab"])
    a = DecoderOracle(SMALL, w)
    b = DecoderOracle(SMALL, w, compute=np.float32, row_invariant=False)
    za, zb = a.prefill(toks), b.prefill(toks)
    np.testing.assert_allclose(zb, za, atol=1e-4)
