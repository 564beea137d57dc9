"""Independent library reference for the oracle pins: transformers' Llama
loaded with the same synthetic weights (float64)."""
import numpy as np
import torch


def llama_config(LlamaConfig, shape, n_layers=None):
    cfg = LlamaConfig(
        vocab_size=shape.vocab, hidden_size=shape.d_model,
        intermediate_size=shape.d_ff,
        num_hidden_layers=n_layers if n_layers is not None else
        shape.n_layers,
        num_attention_heads=shape.n_heads,
        num_key_value_heads=shape.n_kv_heads, head_dim=shape.head_dim,
        rope_theta=shape.rope_theta, rms_norm_eps=shape.norm_eps,
        tie_word_embeddings=False, attention_bias=False, mlp_bias=False,
        max_position_embeddings=1 << 16)
    cfg._attn_implementation = "eager"
    return cfg


_HF_LAYER = {
    "self_attn.q_proj.weight": "wq", "self_attn.k_proj.weight": "wk",
    "self_attn.v_proj.weight": "wv", "self_attn.o_proj.weight": "wo",
    "mlp.gate_proj.weight": "wg", "mlp.up_proj.weight": "wu",
    "mlp.down_proj.weight": "wd", "input_layernorm.weight": "attn_norm",
    "post_attention_layernorm.weight": "mlp_norm",
}


def build(LlamaConfig, LlamaForCausalLM, shape, layer_prefix, n_layers,
          embed, final_norm, lm_head, raw):
    """A float64 LlamaForCausalLM whose layer i holds raw[layer_prefix(i)+*]."""
    m = LlamaForCausalLM(llama_config(LlamaConfig, shape, n_layers))
    m = m.double().eval()
    sd = {"model.embed_tokens.weight": embed, "model.norm.weight": final_norm,
          "lm_head.weight": lm_head}
    for i in range(n_layers):
        for hk, ok in _HF_LAYER.items():
            sd[f"model.layers.{i}.{hk}"] = raw[layer_prefix(i) + ok]
    sd = {k: torch.tensor(np.asarray(v, dtype=np.float64)) for k, v in
          sd.items()}
    missing, unexpected = m.load_state_dict(sd, strict=False)
    assert not unexpected, unexpected
    assert all("rotary" in k for k in missing), missing
    return m


def target_model(hf, shape, tw):
    return build(*hf, shape, lambda i: f"layers.{i}.", shape.n_layers,
                 tw["embed"], tw["final_norm"], tw["lm_head"], tw)


def drafter_trunk(hf, shape, dw, n_layers, embed):
    """The drafter's decoder layers + final norm + LM head as a Llama stack
    (the drafter layers follow the target's architecture)."""
    return build(*hf, shape, lambda i: f"d.layers.{i}.", n_layers, embed,
                 dw["d.final_norm"], dw["d.lm_head"], dw)


@torch.no_grad()
def layer_outputs(model, **kw):
    """Residual stream after every decoder layer, via forward hooks."""
    outs = []
    hooks = [layer.register_forward_hook(
        lambda mod, inp, out: outs.append(
            (out[0] if isinstance(out, tuple) else out).clone()))
        for layer in model.model.layers]
    try:
        logits = model(**kw).logits
    finally:
        for h in hooks:
            h.remove()
    return logits, outs
