"""Pins for the forward-pass oracle.

* An independent implementation: Hugging Face ``transformers`` LlamaForCausalLM in fp64
  (its own RMSNorm, rotate-half RoPE, SwiGLU and grouped-query attention) loaded with the
  same weights; it builds RoPE frequencies in fp32, hence the 1e-6 tolerance.
* Invariants: a block of g+1 rows equals g+1 single-token steps; chunked prefill equals
  one prefill; a zero LM head gives zero logits.
* bf16 rounding against torch's own fp32 -> bfloat16 conversion."""
import numpy as np
import pytest
import torch

from oracle import forward as F
from synth import configs, gen

HF_NAMES = {"wq": "self_attn.q_proj", "wk": "self_attn.k_proj", "wv": "self_attn.v_proj",
            "wo": "self_attn.o_proj", "wg": "mlp.gate_proj", "wu": "mlp.up_proj", "wd": "mlp.down_proj"}


def hf_model(m, w):
    from transformers import LlamaConfig, LlamaForCausalLM
    cfg = LlamaConfig(vocab_size=m.vocab, hidden_size=m.d_model, intermediate_size=m.d_ff,
                      num_hidden_layers=m.n_layers, num_attention_heads=m.n_q_heads,
                      num_key_value_heads=m.n_kv_heads, head_dim=m.head_dim, rms_norm_eps=m.rms_eps,
                      rope_theta=m.rope_base, max_position_embeddings=4096, tie_word_embeddings=False,
                      attention_bias=False, mlp_bias=False)
    torch.manual_seed(0)
    hf = LlamaForCausalLM(cfg).double().eval()
    f64 = lambda a: torch.tensor(F.stored_to_f64(a, m.dtype))
    sd = hf.state_dict()
    with torch.no_grad():
        sd["model.embed_tokens.weight"].copy_(f64(w["embed"]))
        sd["lm_head.weight"].copy_(f64(w["lm_head"]))
        sd["model.norm.weight"].copy_(f64(w["final_norm"]))
        for l in range(m.n_layers):
            for k, n in HF_NAMES.items():
                sd[f"model.layers.{l}.{n}.weight"].copy_(f64(w["layers"][l][k]))
            sd[f"model.layers.{l}.input_layernorm.weight"].copy_(f64(w["layers"][l]["attn_norm"]))
            sd[f"model.layers.{l}.post_attention_layernorm.weight"].copy_(f64(w["layers"][l]["ffn_norm"]))
    return hf


class Unrounded(F.Model):
    """The same oracle with the bf16 storage-rounding points switched off, so that a bf16
    model can be compared with an fp64 reference that does not round."""

    def R(self, x):
        return x


def nonunit_norms(w, m, seed):
    """Random positive norm gains (the workloads use ones) so the pin also covers g."""
    rng = np.random.default_rng(seed)
    conv = (lambda a: a.astype(np.float32)) if m.dtype == "f32" else gen.f32_to_bf16
    for lw in w["layers"]:
        lw["attn_norm"] = conv((0.5 + rng.random(m.d_model)).astype(np.float32))
        lw["ffn_norm"] = conv((0.5 + rng.random(m.d_model)).astype(np.float32))
    w["final_norm"] = conv((0.5 + rng.random(m.d_model)).astype(np.float32))
    return w


@pytest.mark.parametrize("shape", [configs.TINY_F32, configs.TINY_BF16, configs.SMALL_BF16])
def test_matches_hf_llama(synth_built, shape):
    w = nonunit_norms(gen.model_weights(shape, 7), shape, 7)
    om = Unrounded(shape, w)
    B, C, g = 2, [37, 52], [5, 3]
    prompts = [gen.randint(7, 100 + b, C[b], shape.vocab) for b in range(B)]
    cache = F.KVCache(shape, B, 128)
    last, seq_len = F.prefill(om, cache, prompts)
    blocks = [gen.randint(7, 200 + b, g[b] + 1, shape.vocab) for b in range(B)]
    off = np.concatenate([[0], np.cumsum([len(x) for x in blocks])])
    logits, status = F.verify_block(om, cache, seq_len, np.concatenate(blocks), off)
    assert list(status) == [0, 0]
    hf = hf_model(shape, w)
    for b in range(B):
        full = np.concatenate([prompts[b], blocks[b]]).astype(np.int64)
        with torch.no_grad():
            ref = hf(torch.tensor(full[None])).logits[0].numpy()
        scale = np.abs(ref).max()
        assert np.abs(ref[C[b] - 1] - last[b]).max() <= 1e-6 * scale
        assert np.abs(ref[C[b]:] - logits[off[b]:off[b + 1]]).max() <= 1e-6 * scale


@pytest.mark.parametrize("shape", [configs.TINY_F32, configs.TINY_BF16])
def test_block_equals_autoregressive(synth_built, shape):
    w = gen.model_weights(shape, 3)
    om = F.Model(shape, w)
    prompt = gen.randint(3, 1, 20, shape.vocab)
    c1, c2 = F.KVCache(shape, 1, 64), F.KVCache(shape, 1, 64)
    F.prefill(om, c1, [prompt])
    F.prefill(om, c2, [prompt])
    block = gen.randint(3, 2, 6, shape.vocab)
    lb, _ = F.verify_block(om, c1, [20], block, [0, 6])
    for v in range(6):
        lv, _ = F.verify_block(om, c2, [20 + v], block[v:v + 1], [0, 1])
        assert np.abs(lv[0] - lb[v]).max() <= 1e-12 * np.abs(lb).max()
    for l in range(shape.n_layers):
        assert np.array_equal(c1.k[l], c2.k[l]) or np.abs(c1.k[l] - c2.k[l]).max() < 1e-12


def test_chunked_prefill_and_zero_head(synth_built):
    shape = configs.TINY_F32
    w = gen.model_weights(shape, 4)
    om = F.Model(shape, w)
    prompt = gen.randint(4, 1, 30, shape.vocab)
    c1, c2 = F.KVCache(shape, 1, 64), F.KVCache(shape, 1, 64)
    l1, _ = F.verify_block(om, c1, [0], prompt, [0, 30])
    F.verify_block(om, c2, [0], prompt[:11], [0, 11])
    l2, _ = F.verify_block(om, c2, [11], prompt[11:], [0, 19])
    assert np.abs(l1[11:] - l2).max() <= 1e-12 * np.abs(l1).max()
    w0 = dict(w)
    w0["lm_head"] = np.zeros_like(w["lm_head"])
    lz, _ = F.verify_block(F.Model(shape, w0), F.KVCache(shape, 1, 64), [0], prompt[:4], [0, 4])
    assert np.all(lz == 0) and int(np.argmax(lz[0])) == 0


def test_round_bf16_matches_torch():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.normal(size=10000), rng.normal(size=1000) * 1e-30, [0.0, -0.0, 1.0, 3.0e38],
                        # exact ties between two bf16 neighbours: 1 + k*2^-8 + 2^-9
                        1.0 + np.arange(8) * 2.0 ** -7 + 2.0 ** -8]).astype(np.float32).astype(np.float64)
    want = torch.tensor(x, dtype=torch.float32).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(F.round_bf16(x), want)


def test_status_capacity_and_bad_token(synth_built):
    shape = configs.TINY_F32
    om = F.Model(shape, gen.model_weights(shape, 5))
    cache = F.KVCache(shape, 2, 8)
    _, st = F.verify_block(om, cache, [6, 0], [1, 2, 3, 4, shape.vocab], [0, 3, 5])
    assert list(st) == [F.LSV_ERR_CAPACITY, F.LSV_ERR_INVALID_ARG]
    assert np.all(cache.k[0] == 0)
