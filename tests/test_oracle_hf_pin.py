"""Pins the oracle's Llama forward against Hugging Face's independent
implementation (transformers LlamaForCausalLM / LlamaModel in float64).

HF evaluates its rotary angles in float32, so agreement is to ~1e-7
relative; a dropped term, sign or transposed operand shows up at O(1).

This covers the layer math the paper takes from its target family: the
pre-norm RMSNorm, rotate-half RoPE, grouped-query attention, SwiGLU FFN,
final norm and LM head (Sec. 3.1), on the interleaved visual + text input.
"""
import numpy as np
import pytest
import torch

import synth
from synth.configs import MINI_GQA, TINY, ModelDims
from oracle import model as M
from oracle import msd as O

transformers = pytest.importorskip("transformers")


def hf_llama(dims: ModelDims, n_layers=None):
    cfg = transformers.LlamaConfig(
        vocab_size=dims.vocab, hidden_size=dims.d_model, intermediate_size=dims.ffn_dim,
        num_hidden_layers=n_layers or dims.n_layers, num_attention_heads=dims.n_heads,
        num_key_value_heads=dims.n_kv_heads, head_dim=dims.head_dim,
        rms_norm_eps=dims.norm_eps, rope_theta=dims.rope_theta,
        max_position_embeddings=4096, tie_word_embeddings=False,
        attention_bias=False, mlp_bias=False)
    return transformers.LlamaForCausalLM(cfg).double().eval()


def load(m, weights, layers):
    t = lambda a: torch.from_numpy(M.widen(a))
    names = {"wq": "self_attn.q_proj", "wk": "self_attn.k_proj", "wv": "self_attn.v_proj",
             "wo": "self_attn.o_proj", "wg": "mlp.gate_proj", "wu": "mlp.up_proj",
             "wd": "mlp.down_proj", "attn_norm": "input_layernorm",
             "ffn_norm": "post_attention_layernorm"}
    with torch.no_grad():
        m.model.embed_tokens.weight.copy_(t(weights["embed"]))
        m.lm_head.weight.copy_(t(weights["lm_head"]))
        m.model.norm.weight.copy_(t(weights["final_norm"]))
        for l, lw in enumerate(layers):
            layer = m.model.layers[l]
            for k, name in names.items():
                mod = layer.get_submodule(name)
                mod.weight.copy_(t(lw[k]))


@pytest.mark.parametrize("wl", [MINI_GQA, TINY], ids=lambda w: w.name)
def test_prefill_matches_hf(wl):
    dims = wl.dims
    w = synth.make_target_weights(dims, wl.seed)
    tokens, is_visual, visual = synth.make_prompt(wl)
    m = O.Models(dims, w)
    _, first, h, logits = O.prefill(m, tokens, is_visual, visual, wl.prompt_len + 4)
    hf = hf_llama(dims)
    load(hf, w, w["layers"])
    x = M.widen(w["embed"][tokens])
    x[: wl.n_visual] = M.widen(visual)
    with torch.no_grad():
        out = hf(inputs_embeds=torch.from_numpy(x)[None], output_hidden_states=True)
    ref_logits = out.logits[0].numpy()
    ref_h = out.hidden_states[-1][0].numpy()
    scale = np.abs(ref_logits).max()
    assert np.abs(logits - ref_logits).max() <= 2e-6 * scale
    assert np.abs(h - ref_h).max() <= 2e-6 * np.abs(ref_h).max()
    assert first == int(np.argmax(ref_logits[-1]))


def test_draft_layer_matches_hf_decoder_layer():
    wl = TINY
    dims = wl.dims
    w = synth.make_target_weights(dims, wl.seed)
    dr = synth.make_draft_weights(dims, w, wl.seed, "random")
    n = 12
    f = np.random.default_rng(0).standard_normal((n, dims.d_model)) * 0.05
    dkv = M.KVCache(1, n, dims.n_kv_heads, dims.head_dim)
    pos = np.arange(n, dtype=np.int32)
    out = M.draft_forward(dims, dr, dkv, f, pos, pos, 0, n, None)
    hf = hf_llama(dims, n_layers=1)
    load(hf, w, [dr["layer"]])
    captured = {}
    hf.model.layers[0].register_forward_hook(lambda mod, a, o: captured.setdefault(
        "y", o[0] if isinstance(o, tuple) else o))
    with torch.no_grad():
        hf(inputs_embeds=torch.from_numpy(f)[None])
    ref = captured["y"][0].numpy()
    assert np.abs(out - ref).max() <= 2e-6 * np.abs(ref).max()
