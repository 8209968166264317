"""An independent reference decoder: transformers' Qwen2 implementation in
float64, loaded with the synthetic weights (q/k/v biases zeroed, tied
embeddings, the synthetic final-norm gain). Used only to pin the oracle."""
import numpy as np
import torch


def build_qwen2(cfg, w):
    from transformers import Qwen2Config, Qwen2ForCausalLM
    from oracle.numerics import bf16_bits_to_f64
    hc = Qwen2Config(vocab_size=cfg.vocab, hidden_size=cfg.hidden, intermediate_size=cfg.ffn,
                     num_hidden_layers=cfg.n_layers, num_attention_heads=cfg.n_q_heads,
                     num_key_value_heads=cfg.n_kv_heads, rope_theta=cfg.rope_base,
                     rms_norm_eps=cfg.rms_eps, tie_word_embeddings=True,
                     max_position_embeddings=8192)
    torch.manual_seed(0)
    m = Qwen2ForCausalLM(hc).double().eval()

    def t(a):
        a = bf16_bits_to_f64(a) if cfg.wdtype == "bf16" else np.asarray(a, np.float64)
        return torch.from_numpy(np.ascontiguousarray(a))

    with torch.no_grad():
        m.model.embed_tokens.weight.copy_(t(w["embed"]))
        for l, layer in enumerate(m.model.layers):
            p = f"layers.{l}."
            at = layer.self_attn
            at.q_proj.weight.copy_(t(w[p + "wq"]))
            at.k_proj.weight.copy_(t(w[p + "wk"]))
            at.v_proj.weight.copy_(t(w[p + "wv"]))
            at.o_proj.weight.copy_(t(w[p + "wo"]))
            for b in (at.q_proj.bias, at.k_proj.bias, at.v_proj.bias):
                b.zero_()
            layer.mlp.gate_proj.weight.copy_(t(w[p + "w_gate"]))
            layer.mlp.up_proj.weight.copy_(t(w[p + "w_up"]))
            layer.mlp.down_proj.weight.copy_(t(w[p + "w_down"]))
            layer.input_layernorm.weight.copy_(torch.from_numpy(w[p + "attn_norm"].astype(np.float64)))
            layer.post_attention_layernorm.weight.copy_(torch.from_numpy(w[p + "mlp_norm"].astype(np.float64)))
        m.model.norm.weight.copy_(torch.from_numpy(w["final_norm"].astype(np.float64)))
    assert m.lm_head.weight.data_ptr() == m.model.embed_tokens.weight.data_ptr()
    return m
