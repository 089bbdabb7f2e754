"""Pin the oracle's causal decoder against an independent library implementation.

transformers' LlamaForCausalLM (eager attention, float64, CPU) is given the
same weights; its logits must match oracle.causal_forward(rounding=False).
This pins RMSNorm (eps, gain), rotary positions (rotate-half pairing,
theta), multi-head attention, SwiGLU and the final norm / LM head.

transformers computes the rotary angles in float32 even for a float64 model,
so the angle error is about pos * 2**-24 radians; with positions below 64 the
induced logit error stays below 1e-5, which is the tolerance used.
"""

import numpy as np
import pytest
import torch

import oracle
import workloads
from tests.util import oracle_weights

transformers = pytest.importorskip("transformers")


def _hf_model(shape, ow):
    from transformers import LlamaConfig, LlamaForCausalLM

    cfg = LlamaConfig(
        vocab_size=shape.vocab, hidden_size=shape.d_model, intermediate_size=shape.d_ffn,
        num_hidden_layers=shape.n_layers, num_attention_heads=shape.n_heads,
        num_key_value_heads=shape.n_heads, head_dim=shape.head_dim, hidden_act="silu",
        max_position_embeddings=4096, rms_norm_eps=shape.rms_eps,
        rope_parameters={"rope_type": "default", "rope_theta": shape.rope_theta},
        tie_word_embeddings=False, attention_bias=False, mlp_bias=False)
    cfg._attn_implementation = "eager"
    m = LlamaForCausalLM(cfg).to(torch.float64).eval()
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a))
    with torch.no_grad():
        m.model.embed_tokens.weight.copy_(t(ow.tok_embed))
        m.model.norm.weight.copy_(t(ow.final_norm))
        m.lm_head.weight.copy_(t(ow.lm_head))
        for l, layer in enumerate(m.model.layers):
            w = ow.layer(l)
            layer.input_layernorm.weight.copy_(t(w["attn_norm"]))
            layer.post_attention_layernorm.weight.copy_(t(w["ffn_norm"]))
            layer.self_attn.q_proj.weight.copy_(t(w["wq"]))
            layer.self_attn.k_proj.weight.copy_(t(w["wk"]))
            layer.self_attn.v_proj.weight.copy_(t(w["wv"]))
            layer.self_attn.o_proj.weight.copy_(t(w["wo"]))
            layer.mlp.gate_proj.weight.copy_(t(w["wg"]))
            layer.mlp.up_proj.weight.copy_(t(w["wu"]))
            layer.mlp.down_proj.weight.copy_(t(w["wd"]))
    return m


@pytest.mark.parametrize("shape", [
    workloads.MODELS["tiny"],
    # head_dim 128 (the large shapes' head size) on a small stack
    workloads.ModelShape("tiny_dh128", 2, 256, 2, 128, 512, 512, seed=77),
])
def test_causal_forward_matches_transformers_llama(shape):
    ow = oracle_weights(shape, gain_jitter=0.1)
    toks = workloads.draw_tokens(48, shape.vocab, seed=11)
    ours, _, _ = oracle.causal_forward(ow, toks, rounding=False)
    m = _hf_model(shape, ow)
    with torch.no_grad():
        ref = m(torch.from_numpy(toks.astype(np.int64))[None]).logits[0].numpy()
    err = np.abs(ours - ref).max()
    assert err < 1e-5, err
    # the comparison is not vacuous: logits are O(1) and vary across positions
    assert np.abs(ref).max() > 0.5
    assert np.abs(ref[0] - ref[-1]).max() > 0.1
