"""Builds transformers' Qwen3 model (CPU, float64) from the seeded weights, as an
independent library implementation of the target's layer conventions."""
import numpy as np
import torch

from workloads.generate import as_f32


def qwen3_from_weights(wl, W):
    from transformers import Qwen3Config, Qwen3ForCausalLM
    s = wl.target
    cfg = Qwen3Config(vocab_size=s.vocab, hidden_size=s.hidden, intermediate_size=s.ffn,
                      num_hidden_layers=s.n_layers, num_attention_heads=s.n_q_heads,
                      num_key_value_heads=s.n_kv_heads, head_dim=s.head_dim,
                      rope_theta=wl.rope_theta, rms_norm_eps=wl.rms_eps,
                      tie_word_embeddings=False, attn_implementation="eager")
    m = Qwen3ForCausalLM(cfg).double().eval()
    t = lambda n: torch.from_numpy(as_f32(W[n]).astype(np.float64))
    sd = {"model.embed_tokens.weight": t("embed"), "model.norm.weight": t("target.final_norm"),
          "lm_head.weight": t("lm_head")}
    names = [("self_attn.q_proj", "q_proj"), ("self_attn.k_proj", "k_proj"),
             ("self_attn.v_proj", "v_proj"), ("self_attn.o_proj", "o_proj"),
             ("self_attn.q_norm", "q_norm"), ("self_attn.k_norm", "k_norm"),
             ("input_layernorm", "input_norm"), ("post_attention_layernorm", "post_norm"),
             ("mlp.gate_proj", "gate_proj"), ("mlp.up_proj", "up_proj"),
             ("mlp.down_proj", "down_proj")]
    for l in range(s.n_layers):
        for a, b in names:
            sd[f"model.layers.{l}.{a}.weight"] = t(f"target.{l}.{b}")
    m.load_state_dict(sd, strict=True)
    return m


def hf_logits(model, tokens):
    with torch.no_grad():
        ids = torch.from_numpy(np.asarray(tokens, dtype=np.int64))[None]
        return model(ids).logits[0].numpy()
