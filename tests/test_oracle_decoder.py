"""Pins of the oracle's forward pass against things other than itself.

* a library implementation of the same decoder (HuggingFace ``LlamaForCausalLM``,
  float64, eager attention) on a small fp32 shape with random gains;
* library routines for RMSNorm, RoPE and bf16 rounding (torch);
* the paper's statement that one verify pass over d+1 positions yields the
  autoregressive conditionals (Sec. III-B, Algorithm 1): verify logits equal
  d+1 sequential single-token decodes and a from-scratch recompute;
* RoPE invariants: norm preservation and dependence on relative position only;
* grouped-query attention: the library decoder with fewer K/V heads, and the
  special case it reduces to -- multi-head attention whose K/V projections
  repeat each K/V head's rows for every query head of its group.
"""

import numpy as np
import pytest
import torch

from oracle.decoder import (Decoder, apply_rope, bf16_round, rms_norm, rope_tables)
from synth import ModelWeights
from synth.configs import ModelShape

pytestmark = pytest.mark.filterwarnings("ignore::UserWarning")


def _model(shape, seed=7, keep=True):
    mw = ModelWeights(shape, seed)
    return Decoder(shape, mw.get, keep_f64=keep), mw


SMALL_F32 = ModelShape("t-f32", n_layers=2, d_model=64, n_heads=2, head_dim=32, d_ffn=96,
                       vocab=97, weight_dtype="f32", kv_dtype="f32", init_std=0.08, gain_std=0.2)
SMALL_GQA = ModelShape("t-gqa", n_layers=2, d_model=128, n_heads=4, head_dim=32, d_ffn=96,
                       vocab=97, weight_dtype="f32", kv_dtype="f32", init_std=0.08, gain_std=0.2,
                       n_kv_heads=2, rope_theta=500000.0)
SMALL_BF16 = ModelShape("t-bf16", n_layers=2, d_model=128, n_heads=2, head_dim=64, d_ffn=256,
                        vocab=211, weight_dtype="bf16", kv_dtype="bf16", init_std=0.05, gain_std=0.2)


def test_rmsnorm_matches_torch():
    rng = np.random.default_rng(0)
    x = rng.standard_normal((5, 48)) * 3
    g = rng.standard_normal(48)
    ref = torch.nn.functional.rms_norm(torch.from_numpy(x), (48,), torch.from_numpy(g), eps=1e-5)
    np.testing.assert_allclose(rms_norm(x, g, 1e-5), ref.numpy(), rtol=1e-12, atol=1e-12)


def test_rope_matches_hf_and_invariants():
    from transformers.models.llama.modeling_llama import apply_rotary_pos_emb
    rng = np.random.default_rng(1)
    hd, H = 64, 3
    pos = np.array([0, 1, 5, 77, 1023, 4000])
    q = rng.standard_normal((len(pos), H, hd))
    cos, sin = rope_tables(pos, hd, 10000.0)
    out = apply_rope(q, cos, sin)
    # HF convention: cos/sin repeated over both halves, rotate_half pairing.
    c = torch.from_numpy(np.concatenate([cos, cos], -1))
    s = torch.from_numpy(np.concatenate([sin, sin], -1))
    qt = torch.from_numpy(q)
    ref, _ = apply_rotary_pos_emb(qt, qt, c, s, unsqueeze_dim=1)
    np.testing.assert_allclose(out, ref.numpy(), rtol=1e-12, atol=1e-12)
    # position 0 is the identity, norms are preserved
    np.testing.assert_allclose(out[0], q[0], atol=1e-15)
    np.testing.assert_allclose(np.linalg.norm(out, axis=-1), np.linalg.norm(q, axis=-1), rtol=1e-12)
    # q.k depends on the position difference only
    a, b = rng.standard_normal(hd), rng.standard_normal(hd)
    def dot(m, n):
        cm, sm = rope_tables(np.array([m]), hd, 10000.0)
        cn, sn = rope_tables(np.array([n]), hd, 10000.0)
        return float(apply_rope(a[None, None], cm, sm).ravel() @ apply_rope(b[None, None], cn, sn).ravel())
    assert abs(dot(10, 3) - dot(107, 100)) < 1e-10
    assert abs(dot(10, 3) - dot(10, 4)) > 1e-6


def test_bf16_round_matches_torch_and_ties():
    rng = np.random.default_rng(2)
    x = np.concatenate([rng.standard_normal(10000) * 10.0 ** rng.integers(-6, 6, 10000),
                        [1.0, 1 + 2 ** -8, 1 + 3 * 2 ** -8, -1 - 2 ** -8, 0.0, -0.0]])
    ref = torch.from_numpy(x.astype(np.float32)).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(bf16_round(x), ref)
    assert bf16_round(np.array([1 + 2 ** -8]))[0] == 1.0  # tie -> even mantissa
    assert bf16_round(np.array([1 + 3 * 2 ** -8]))[0] == 1 + 2 ** -6


def _hf_model(shape, mw):
    from transformers import LlamaConfig, LlamaForCausalLM
    cfg = LlamaConfig(vocab_size=shape.vocab, hidden_size=shape.d_model,
                      intermediate_size=shape.d_ffn, num_hidden_layers=shape.n_layers,
                      num_attention_heads=shape.n_heads, num_key_value_heads=shape.kv_heads,
                      head_dim=shape.head_dim, rms_norm_eps=shape.rms_eps,
                      rope_theta=shape.rope_theta, max_position_embeddings=512,
                      tie_word_embeddings=False, attention_bias=False, mlp_bias=False)
    cfg._attn_implementation = "eager"
    m = LlamaForCausalLM(cfg).double().eval()
    f = lambda a: torch.from_numpy(np.asarray(a, dtype=np.float64))
    sd = {"model.embed_tokens.weight": f(mw.get("embed")), "lm_head.weight": f(mw.get("lm_head")),
          "model.norm.weight": f(mw.get("g_final"))}
    names = {"wq": "self_attn.q_proj", "wk": "self_attn.k_proj", "wv": "self_attn.v_proj",
             "wo": "self_attn.o_proj", "wg": "mlp.gate_proj", "wu": "mlp.up_proj",
             "wd": "mlp.down_proj"}
    for l in range(shape.n_layers):
        for k, n in names.items():
            sd[f"model.layers.{l}.{n}.weight"] = f(mw.get(k, l))
        sd[f"model.layers.{l}.input_layernorm.weight"] = f(mw.get("g_attn", l))
        sd[f"model.layers.{l}.post_attention_layernorm.weight"] = f(mw.get("g_ffn", l))
    m.load_state_dict(sd, strict=False)
    return m


@pytest.mark.parametrize("shape", [SMALL_F32, SMALL_GQA], ids=lambda s: s.name)
def test_decoder_matches_hf_llama(shape):
    dec, mw = _model(shape)
    hf = _hf_model(shape, mw)
    rng = np.random.default_rng(3)
    toks = rng.integers(0, shape.vocab, 40)
    with torch.no_grad():
        ref = hf(torch.from_numpy(toks)[None]).logits[0].numpy()
    cache = dec.new_cache(64)
    dec.prefill(cache, toks[:33])  # cached prefix, then a 7-row verify block
    out = dec.forward(cache, toks[33:])
    # HF computes the RMSNorm and the RoPE angles in float32, hence the tolerance.
    assert np.abs(out - ref[33:]).max() < 2e-5
    assert np.abs(ref).max() > 0.5  # the comparison is not trivially small


def test_gqa_equals_mha_with_repeated_kv_heads():
    from dataclasses import replace
    gqa, mw = _model(SMALL_GQA)
    G = SMALL_GQA.n_heads // SMALL_GQA.kv_heads
    hd = SMALL_GQA.head_dim

    def get_mha(kind, layer=None):
        t = mw.get(kind, layer)
        if kind in ("wk", "wv"):  # [KVH*hd, d] -> [H*hd, d], K/V head j serves query heads jG..jG+G-1
            t = np.repeat(t.reshape(SMALL_GQA.kv_heads, hd, -1), G, axis=0).reshape(SMALL_GQA.n_heads * hd, -1)
        return t

    mha_shape = replace(SMALL_GQA, n_kv_heads=0)
    mha = Decoder(mha_shape, get_mha, keep_f64=True)
    rng = np.random.default_rng(8)
    toks = rng.integers(0, SMALL_GQA.vocab, 36)
    c1, c2 = gqa.new_cache(48), mha.new_cache(48)
    gqa.prefill(c1, toks[:30])
    mha.prefill(c2, toks[:30])
    a, b = gqa.forward(c1, toks[30:]), mha.forward(c2, toks[30:])
    np.testing.assert_allclose(a, b, rtol=0, atol=1e-12)
    assert c1.k[0].shape[0] == SMALL_GQA.kv_heads and c2.k[0].shape[0] == SMALL_GQA.n_heads
    # a genuinely different model if the K/V heads are paired with the wrong query heads
    def get_wrong(kind, layer=None):
        t = get_mha(kind, layer)
        if kind in ("wk", "wv"):
            t = t.reshape(SMALL_GQA.n_heads, hd, -1)[::-1].reshape(SMALL_GQA.n_heads * hd, -1)
        return t
    wrong = Decoder(mha_shape, get_wrong, keep_f64=True)
    c3 = wrong.new_cache(48)
    wrong.prefill(c3, toks[:30])
    assert np.abs(wrong.forward(c3, toks[30:]) - a).max() > 1e-3


@pytest.mark.parametrize("shape", [SMALL_F32, SMALL_BF16, SMALL_GQA], ids=lambda s: s.name)
def test_verify_block_equals_sequential_decodes(shape):
    dec, _ = _model(shape)
    rng = np.random.default_rng(4)
    toks = rng.integers(0, shape.vocab, 30)
    c1 = dec.new_cache(40)
    dec.prefill(c1, toks[:24])
    block = dec.forward(c1, toks[24:])
    c2 = dec.new_cache(40)
    dec.prefill(c2, toks[:24])
    seq = np.stack([dec.forward(c2, toks[i:i + 1])[0] for i in range(24, 30)])
    np.testing.assert_allclose(block, seq, rtol=0, atol=1e-11)
    for l in range(shape.n_layers):
        np.testing.assert_array_equal(c1.k[l][:, :30], c2.k[l][:, :30])


@pytest.mark.parametrize("shape", [SMALL_F32, SMALL_BF16])
def test_verify_block_equals_full_recompute(shape):
    dec, _ = _model(shape)
    rng = np.random.default_rng(5)
    toks = rng.integers(0, shape.vocab, 50)
    c1 = dec.new_cache(64)
    dec.prefill(c1, toks[:41])
    block = dec.forward(c1, toks[41:])
    c2 = dec.new_cache(64)
    full = dec.forward(c2, toks)
    np.testing.assert_allclose(block, full[41:], rtol=0, atol=1e-11)


def test_bf16_kv_storage_is_what_attention_reads():
    dec, _ = _model(SMALL_BF16)
    c = dec.new_cache(16)
    dec.forward(c, np.arange(5))
    for l in range(SMALL_BF16.n_layers):
        np.testing.assert_array_equal(bf16_round(c.k[l]), c.k[l])
        np.testing.assert_array_equal(bf16_round(c.v[l]), c.v[l])


@pytest.mark.parametrize("shape", [SMALL_BF16, SMALL_GQA], ids=["bf16", "gqa"])
def test_forward_many_equals_forward_per_request(shape):
    """The layer-by-layer driver over several requests (used to generate the
    stored oracle results of the large batched workloads) gives every request
    exactly what ``forward`` gives it alone: prefill, a one-token step and a
    multi-row block, with ragged lengths."""
    dec, _ = _model(shape, seed=11)
    rng = np.random.default_rng(12)
    lens = [1, 17, 40]
    prompts = [rng.integers(0, shape.vocab, size=L) for L in lens]
    solo = [dec.new_cache(64) for _ in lens]
    many = [dec.new_cache(64) for _ in lens]
    for c, p in zip(solo, prompts):
        dec.forward(c, p, want_logits=False)
    dec.forward_many(many, prompts, want_logits=False)
    for step in ([5], [3, 9, 11, 2]):
        toks = [np.array(step) + b for b in range(len(lens))]
        ref = [dec.forward(c, t) for c, t in zip(solo, toks)]
        got = dec.forward_many(many, toks)
        for r, g in zip(ref, got):
            np.testing.assert_array_equal(r, g)
    for cs, cm in zip(solo, many):
        assert cs.length == cm.length
        for l in range(shape.n_layers):
            np.testing.assert_array_equal(cs.k[l], cm.k[l])
            np.testing.assert_array_equal(cs.v[l], cm.v[l])


def test_bf16_widening_matches_torch_for_every_pattern():
    """bf16 -> float64 widening of all 65536 bit patterns equals torch's
    bfloat16 -> float64 conversion (NaN patterns stay NaN)."""
    from oracle.decoder import bf16_bits_to_f64
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    with np.errstate(invalid="ignore"):  # NaN patterns
        got = bf16_bits_to_f64(bits)
    ref = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).to(torch.float64).numpy()
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(got), nan)
    np.testing.assert_array_equal(got[~nan], ref[~nan])
    assert np.array_equal(np.signbit(got[~nan]), np.signbit(ref[~nan]))
